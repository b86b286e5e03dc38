/*
 * purlin.h -- C ABI of an MI355X (gfx950) datapath executor for collectives.
 *
 * The operations follow "Purlin: Separating Orchestration from the Datapath
 * of Collectives" (arXiv 2609.36954):
 *
 *   - collective semantics: Section 2.1 ("Stable communication semantics");
 *   - collectives as layout transformations with a consume op (copy or
 *     reduce) between packed / scattered / transposed layouts, and
 *     AllReduce = compose<ReduceScatter, AllGather>: Section 3.1, Listing 1;
 *   - chunk-level consumption and its address rule (packed output: dst +
 *     offset; scattered/transposed output: dst + peer * partBytes + offset):
 *     Section 3.2, Listing 2;
 *   - copy and reduce of the datapath, the reduction summing in FP32 in
 *     ascending rank order from zero (Eq. 2): Section 3.3, Listing 3.
 *
 * On one GPU, the P ranks of a collective are P separate device buffers.  A
 * host-side planner (purlin_plan) turns (op, P, count, dtype, chunk) into a
 * table of chunk descriptors; purlin_exec binds 2P buffer pointers and runs
 * the table with hand-written HIP kernels.  purlin_pack / purlin_unpack are
 * the MoE dispatch and combine of expert parallelism (Section 2, Table 2).
 *
 * Conventions shared by every entry point:
 *   - Status codes only: nothing throws or aborts across this ABI.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     call that returns anything but PURLIN_OK has enqueued nothing.
 *   - Device work is asynchronous on the given stream (a hipStream_t passed
 *     as void*; NULL = the default stream).  The caller owns every data
 *     buffer and keeps it alive until the stream has finished with it.
 *   - Device pointers must be 16-byte aligned.
 *   - bf16 data is the 16-bit encoding (upper half of a binary32 encoding).
 */
#ifndef PURLIN_H
#define PURLIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define PURLIN_API __attribute__((visibility("default")))
#else
#define PURLIN_API
#endif

typedef enum purlin_status {
    PURLIN_OK = 0,
    PURLIN_ERR_INVALID = 1,     /* a bad argument; nothing was enqueued */
    PURLIN_ERR_UNSUPPORTED = 2, /* valid request the library does not implement */
    PURLIN_ERR_NOMEM = 3,       /* descriptor table too large, or an allocation failed */
    PURLIN_ERR_DEVICE = 4       /* a HIP call or kernel launch failed */
} purlin_status;

/* Collectives (Section 2.1; Listing 1 gives consume op and layouts):
 *   ALLREDUCE      reduce, scattered -> scattered  (compose<RS, AG>)
 *   REDUCE_SCATTER reduce, scattered -> packed
 *   ALLGATHER      copy,   packed    -> scattered
 *   ALLTOALL       copy,   scattered -> transposed
 * Rooted collectives (Appendix A), planned with purlin_plan_rooted:
 *   BROADCAST      the root's input to every rank   (compose<scatter, AG>)
 *   REDUCE         every rank's input reduced at the root
 *                                                   (compose<RS, gather>)
 *   SCATTER        copy, scattered -> packed, only the root produces
 *   GATHER         copy, packed -> scattered, only the root consumes      */
typedef enum purlin_op {
    PURLIN_ALLREDUCE = 0,
    PURLIN_REDUCE_SCATTER = 1,
    PURLIN_ALLGATHER = 2,
    PURLIN_ALLTOALL = 3,
    PURLIN_BROADCAST = 4,
    PURLIN_REDUCE = 5,
    PURLIN_SCATTER = 6,
    PURLIN_GATHER = 7,
    /* Variable-size collectives (Section 3.1: the V layouts take partition
     * sizes at run time), planned with purlin_plan_v, run with purlin_exec_v */
    PURLIN_ALLGATHERV = 8,      /* copy,   packedV    -> scatteredV  */
    PURLIN_REDUCE_SCATTERV = 9, /* reduce, scatteredV -> packedV     */
    PURLIN_ALLTOALLV = 10       /* copy,   scatteredV -> transposedV */
} purlin_op;

typedef enum purlin_dtype { PURLIN_FP32 = 0, PURLIN_BF16 = 1 } purlin_dtype;

/* Consume op of a descriptor (Section 3.1, "copy" and "reduce"). */
typedef enum purlin_kind { PURLIN_KIND_COPY = 0, PURLIN_KIND_REDUCE = 1 } purlin_kind;

/* One chunk descriptor (64 bytes).  Buffer indices refer to the bufs[]
 * array given to purlin_exec: bufs[0..P-1] are the inputs in_0..in_{P-1},
 * bufs[P..2P-1] the outputs out_0..out_{P-1}.
 *
 *   COPY:   for every destination j < ndst:
 *             bufs[dst_buf + j*dst_step][dst_off .. +bytes) =
 *             bufs[src_buf][src_off .. +bytes)                  (bit copy)
 *   REDUCE: for every element i of the byte range and every j < ndst:
 *             acc = +0.0f;
 *             for p = 0 .. nsrc-1: acc += widen(bufs[src_buf + p*src_step][src_off + i]);
 *             bufs[dst_buf + j*dst_step][dst_off + i] = narrow(acc)
 *           in binary32, round to nearest even, no flush of denormals
 *           (Eq. 2); widen/narrow are the identity for fp32 and exact
 *           widening / round-to-nearest-even narrowing for bf16.
 *
 * phase: descriptors of phase 1 start only after every descriptor of phase
 * 0 has completed (stream order between two launches).  A multi-destination
 * descriptor (ndst > 1) reads its sources once and writes every destination. */
typedef struct purlin_desc {
    uint32_t kind;     /* purlin_kind */
    uint32_t phase;    /* 0 or 1 */
    uint32_t nsrc;     /* 1 for COPY; number of summed sources for REDUCE */
    uint32_t src_buf;  /* bufs[] index of source 0 */
    uint32_t src_step; /* bufs[] index stride between successive sources */
    uint32_t ndst;     /* number of destinations written */
    uint32_t dst_buf;  /* bufs[] index of destination 0 */
    uint32_t dst_step; /* bufs[] index stride between successive destinations */
    uint64_t src_off;  /* byte offset into every source */
    uint64_t dst_off;  /* byte offset into every destination */
    uint64_t bytes;    /* length in bytes (a multiple of the element size) */
    uint32_t part;     /* partition k the range belongs to */
    uint32_t chunk;    /* chunk c within the partition */
} purlin_desc;

/* Planning policy (the paper's codesign policies, Section 3.2/3.3): how the
 * descriptors are split into work items and how AllGather / AllReduce are
 * scheduled.  Zero in a field means "choose automatically". */
typedef struct purlin_policy {
    uint64_t item_bytes; /* bytes of one work item (a multiple of 16; 0 = auto) */
    uint32_t fanout;     /* 0 auto, 1 = one COPY descriptor per destination,
                            2 = one multi-destination COPY per source chunk   */
    uint32_t ar_mode;    /* AllReduce: 0 auto, 1 = two phases (ReduceScatter
                            into out_k's partition k, then copies of it to
                            every other rank: the in-place compose of
                            Section 3.1), 2 = one phase (each chunk reduced
                            once and written to all P outputs), 3 = the two
                            phases of 1 in one launch: a chunk's copies start
                            when its reduction has finished (per-chunk
                            counters with epochs, Section 3.2 and 4.2; such a
                            plan must not run concurrently with itself).
                            Mode 3 demonstrates the in-kernel notify/consume:
                            it is never chosen automatically and measured
                            slower than mode 1 at every size on MI355X
                            (P = 8, bf16: 1.08x its time at 256 MiB per
                            rank, 1.4x at 32 MiB, 2.8x at 2 MiB). */
    uint32_t load_hint;  /* global loads:  0 auto, 1 cached, 2 non-temporal */
    uint32_t store_hint; /* global stores: 0 auto, 1 cached, 2 non-temporal
                            (variable-size plans apply one setting to loads
                            and stores: non-temporal if either hint is) */
    uint32_t max_workgroups; /* 0 = one wavefront per work item; otherwise every
                            launch of the plan has at most this many 256-thread
                            workgroups (4 wavefronts each) and its wavefronts
                            stride over the items: the collective runs on a
                            bounded share of the GPU's 256 CUs, leaving the
                            rest to overlapped compute (the paper's
                            resource-constrained execution, Section 5).  Not
                            with ar_mode 3 (PURLIN_ERR_UNSUPPORTED). */
    uint32_t copy_depth; /* copy phases of the fixed-size and rooted
                            collectives: 16-byte loads each lane keeps in flight
                            before it stores (the pipeline depth of Section
                            3.3 / Eq. 1: bytes in flight per wavefront =
                            copy_depth * 1 KiB); 0 = auto (8 on a grid capped
                            at 128 workgroups or fewer, else 4), or 1, 2, 4, 8 */
    uint32_t reserved[3];/* must be zero */
} purlin_policy;

#define PURLIN_PLAN_HOST_ONLY 1u /* build the tables on the host only (no device
                                    upload); such a plan can be inspected but
                                    not executed */
#define PURLIN_PLAN_SHARE_PUSH 4u /* purlin_plan_share only: the rank's push
                                    share (the descriptors that read its
                                    input) instead of its pull share */
#define PURLIN_PLAN_COUNTS_TRANSPOSED 2u /* ALLTOALLV only: read the P x P
                                    sizes column-major, counts[r*P + p] =
                                    what rank p sends to rank r.  The reverse
                                    exchange of an expert-parallel dispatch
                                    (the combine, Table 2) then reuses the
                                    dispatch's counts as they are. */

#define PURLIN_MAX_RANKS 16
#define PURLIN_MAX_ITEMS (1ull << 24)

typedef struct purlin_plan_s* purlin_plan_t;

/* Build a plan for a non-rooted `op` (ALLREDUCE, REDUCE_SCATTER, ALLGATHER,
 * ALLTOALL) over P ranks (1..16) of `count` elements per rank
 * on the scattered side (the paper's message-size convention, Section 5
 * "Microbenchmark methodology"):
 *     ALLREDUCE      in: count      out: count        elements per rank
 *     REDUCE_SCATTER in: count      out: count / P
 *     ALLGATHER      in: count / P  out: count
 *     ALLTOALL       in: count      out: count
 * `count` must be a multiple of P (uniform slices, Section 2.1); count = 0
 * is a valid plan whose exec is a no-op.  `chunk_bytes` (>= element size and
 * a multiple of it) is the chunk of Section 3.2: every partition of M =
 * count/P elements is cut into ceil(M*s / chunk_bytes) chunks, the last one
 * possibly shorter; the result does not depend on it.
 * The plan owns a host descriptor table and its device copy (uploaded
 * synchronously here, once).  Errors: PURLIN_ERR_INVALID (bad op, dtype,
 * P, count, chunk, null out_plan), PURLIN_ERR_NOMEM (more than
 * PURLIN_MAX_ITEMS work items, or an allocation failed), PURLIN_ERR_DEVICE
 * (the device upload failed).  *out_plan is NULL on error. */
PURLIN_API purlin_status purlin_plan(purlin_op op, int P, uint64_t count, purlin_dtype dtype,
                          uint64_t chunk_bytes, purlin_plan_t* out_plan);

/* A rooted collective (Appendix A) with root rank `root` (0 <= root < P).
 * `count` is the root-side scattered size N (a multiple of P):
 *     BROADCAST  in: N (root only)      out: N       on every rank
 *     REDUCE     in: N on every rank    out: N       (root only)
 *     SCATTER    in: N (root only)      out: N / P   on every rank
 *     GATHER     in: N / P on every rank out: N      (root only)
 * Buffers a rank does not use (the inputs of non-roots for BROADCAST and
 * SCATTER, the outputs of non-roots for REDUCE and GATHER) are ignored by
 * purlin_exec and may be NULL.  Policy, flags and errors as for
 * purlin_plan_ex; PURLIN_ERR_INVALID also for a root out of range or a
 * non-rooted op. */
PURLIN_API purlin_status purlin_plan_rooted(purlin_op op, int P, int root, uint64_t count, purlin_dtype dtype,
                                            uint64_t chunk_bytes, const purlin_policy* policy, uint32_t flags,
                                            purlin_plan_t* out_plan);

/* Rank `rank`'s share of a collective run on P GPUs: the descriptors of the
 * full plan that write out_rank, each narrowed to that one destination.
 * Every rank pulls what it consumes (Section 3.2: a consumer reads its
 * peers' chunks), so on P GPUs each one would execute its own share, with
 * the other ranks' buffers reached as peer memory; on one GPU the share is
 * one rank's work at its real shape.
 *   REDUCE_SCATTER  partition `rank` of every input reduced into out_rank
 *   ALLGATHER       every rank's input copied into out_rank
 *   ALLTOALL        partition `rank` of every input into out_rank
 *   ALLREDUCE       compose<RS, AG>: phase 0 reduces partition `rank` into
 *                   out_rank, phase 1 copies partition k of out_k into
 *                   out_rank for k != rank (it reads what rank k's share
 *                   wrote in its phase 0).  ar_mode 0 selects this form;
 *                   ar_mode 2 has the rank reduce every partition itself;
 *                   ar_mode 3 gives PURLIN_ERR_UNSUPPORTED.
 *   rooted ops      as the full plan, restricted to out_rank (empty for a
 *                   REDUCE or GATHER share of a rank that is not the root)
 * `root` is -1 for the non-rooted collectives and the root rank for the
 * rooted ones.  The share reads and writes only the buffers its
 * descriptors name (purlin_exec checks those; the others may be NULL) and
 * writes out_rank and nothing else.  The P shares together write exactly
 * what the full plan writes.
 * With PURLIN_PLAN_SHARE_PUSH in `flags` the share is instead the
 * descriptors that read in_rank, unchanged (multi-destination copies keep
 * every destination): the rank pushes its data into the others' outputs.
 * Push applies to the collectives made of copies only (ALLGATHER,
 * ALLTOALL, BROADCAST, SCATTER, GATHER; empty for a BROADCAST or SCATTER
 * share of a rank that is not the root); a reduction needs every rank's
 * data in one place, so ALLREDUCE, REDUCE_SCATTER and REDUCE give
 * PURLIN_ERR_UNSUPPORTED.  The P push shares together are the full plan.
 * Other arguments and errors as purlin_plan_ex and purlin_plan_rooted;
 * PURLIN_ERR_INVALID also for rank outside [0, P) or a variable-size op. */
PURLIN_API purlin_status purlin_plan_share(purlin_op op, int P, int root, int rank, uint64_t count,
                                           purlin_dtype dtype, uint64_t chunk_bytes, const purlin_policy* policy,
                                           uint32_t flags, purlin_plan_t* out_plan);

/* A variable-size collective over P ranks: every input buffer holds
 * `in_capacity` elements and every output buffer `out_capacity`.  The sizes
 * are not part of the plan: purlin_exec_v reads them from device memory at
 * run time, so they may be produced by an earlier kernel on the stream (e.g.
 * purlin_pack's dest_counts, with unit = the row length) and the call can be
 * captured in a graph.  Counts are in units of `unit` elements
 * (1 <= unit <= 2^31).  `chunk_bytes` cuts a virtual index space into
 * chunks, as for the fixed-size plans: the gathered output (ALLGATHERV,
 * out_capacity), the partitioned input (REDUCE_SCATTERV, in_capacity), or
 * for ALLTOALLV each destination's output (descriptor part = r, dst_buf =
 * out_r) or, when in_capacity < out_capacity, each source's input (part =
 * p, src_buf = in_p, dst_step = 1: the sizes pick the output).  Covering the
 * smaller side keeps a receive buffer sized for the worst case (P*T*K rows
 * of an expert-parallel dispatch) from adding idle work items.  Policy and errors as for
 * purlin_plan_ex; flags: PURLIN_PLAN_HOST_ONLY, and for ALLTOALLV
 * PURLIN_PLAN_COUNTS_TRANSPOSED.  PURLIN_ERR_INVALID also for a non-V op, a
 * bad unit or a flag the op does not take. */
PURLIN_API purlin_status purlin_plan_v(purlin_op op, int P, uint64_t in_capacity, uint64_t out_capacity,
                                       purlin_dtype dtype, uint64_t chunk_bytes, uint64_t unit,
                                       const purlin_policy* policy, uint32_t flags, purlin_plan_t* out_plan);

/* Run a variable-size plan.  `counts` is device memory (int32):
 *   ALLGATHERV      counts[p], p < P: elements rank p contributes; every
 *                   out_r receives them in rank order,
 *                   out_r[off_p + i] = in_p[i], off_p = sum(counts[0..p)).
 *   REDUCE_SCATTERV counts[r]: partition sizes of every input; out_r[i] =
 *                   rank-order sum (Eq. 2) of in_p[off_r + i], i < counts[r].
 *   ALLTOALLV       counts[p*P + r]: elements rank p sends to rank r
 *                   (counts[r*P + p] with PURLIN_PLAN_COUNTS_TRANSPOSED);
 *                   in_p holds them in destination order, out_r receives
 *                   them in source order.
 * Each count (times unit) must be >= 0, every input's part must fit
 * in_capacity and every output's part out_capacity; otherwise the call
 * writes nothing and, if `dev_status` (device int32, optional) is given,
 * sets it to 1 (else 0).  One launch of a fixed number of wavefronts that
 * stride over the work items below the run-time sizes, so capacity left
 * unused costs no work.  A plan of zero capacity ignores bufs, which may
 * then be NULL (the sizes are still checked when dev_status is given).
 * Host-side errors as for purlin_exec, plus PURLIN_ERR_INVALID for a non-V
 * plan or NULL counts.
 * purlin_exec rejects V plans. */
PURLIN_API purlin_status purlin_exec_v(purlin_plan_t plan, void* const* bufs, const int32_t* counts,
                                       int32_t* dev_status, void* stream);

/* purlin_plan with an explicit policy (NULL = automatic) and flags
 * (0 or PURLIN_PLAN_HOST_ONLY).  PURLIN_ERR_INVALID also for a policy with
 * item_bytes not a multiple of 16, fanout > 2, ar_mode > 3, a hint > 2 or
 * nonzero reserved fields, and for unknown flags.  Hints change only how
 * the caches treat the streams, never the result. */
PURLIN_API purlin_status purlin_plan_ex(purlin_op op, int P, uint64_t count, purlin_dtype dtype,
                             uint64_t chunk_bytes, const purlin_policy* policy, uint32_t flags,
                             purlin_plan_t* out_plan);

/* Sizes of a plan (any output pointer may be NULL):
 *   n_desc             chunk descriptors;
 *   in_bytes_per_rank  bytes each used bufs[p], p < P, must hold;
 *   out_bytes_per_rank bytes each used bufs[P + r] must hold;
 *   sched_bytes        bytes the schedule reads plus writes,
 *                      sum over descriptors of (nsrc + ndst) * bytes. */
PURLIN_API purlin_status purlin_plan_info(purlin_plan_t plan, uint64_t* n_desc, uint64_t* in_bytes_per_rank,
                               uint64_t* out_bytes_per_rank, uint64_t* sched_bytes);

/* The chunk descriptor table (host memory owned by the plan, valid until
 * purlin_plan_destroy): *n entries of *stride bytes each, phase 0 first. */
PURLIN_API purlin_status purlin_plan_descriptors(purlin_plan_t plan, const purlin_desc** table, uint64_t* n,
                                      uint64_t* stride);

/* The work items the kernels execute: the descriptors cut at item_bytes
 * boundaries, one item per wavefront (host copy, owned by the plan).
 * phase_begin[0..2] (optional, may be NULL) receives the first item of
 * phase 0, of phase 1, and the item count. */
PURLIN_API purlin_status purlin_plan_items(purlin_plan_t plan, const purlin_desc** items, uint64_t* n,
                                uint64_t phase_begin[3]);

/* Run the plan (Section 3.2, Listing 2: every chunk descriptor is consumed
 * by its copy or reduce op, Section 3.3, Listing 3 and Eq. 2, at the
 * address the layout rule gives; an AllReduce runs its ReduceScatter phase
 * before its AllGather phase, Section 3.1).
 * bufs[] holds 2P device pointers, in_0..in_{P-1} then
 * out_0..out_{P-1}, sized per purlin_plan_info (entries a rooted plan does
 * not use are ignored).  Each phase is one kernel
 * launch on `stream`; no host-device copy, no allocation, no
 * synchronisation (graph-capturable).  Errors (nothing enqueued):
 * PURLIN_ERR_INVALID for a NULL or host-only plan, NULL bufs, a NULL or
 * misaligned pointer, an input range overlapping an output range other
 * than an in-place pair (below), or two output ranges overlapping;
 * PURLIN_ERR_DEVICE if a launch fails.  Inputs may alias each other.
 * In place: a rank's input and output may be one buffer in the layouts
 * where every element is read before it is rewritten by the same
 * wavefront (or by a later phase):
 *     ALLREDUCE, BROADCAST, REDUCE   in_r == out_r
 *     REDUCE_SCATTER, SCATTER        out_r == in_r + r * out_bytes_per_rank
 *     ALLGATHER, GATHER              in_r == out_r + r * in_bytes_per_rank
 * (rooted ops: the root's own pair only; the pointers must still be
 * 16-byte aligned, so an offset of r partitions needs out_bytes_per_rank
 * resp. in_bytes_per_rank to be a multiple of 16); not ALLTOALL, not the
 * variable-size collectives.  For count = 0 it returns PURLIN_OK and
 * ignores bufs.  A plan is immutable: concurrent execs on different
 * streams with distinct buffers are safe (except for a single-launch
 * AllReduce plan, ar_mode 3, whose per-chunk counters belong to the plan:
 * run it on one stream at a time). */
PURLIN_API purlin_status purlin_exec(purlin_plan_t plan, void* const* bufs, void* stream);

/* Device error word of a plan (0 = none).  Only single-launch AllReduce
 * plans (ar_mode 3) can set it: a copy that waited longer than a fixed bound
 * for its chunk gives up and sets it, so a launch always completes.
 * Synchronous: waits for all work queued on the device (a device-wide
 * synchronisation), then reads the word. */
PURLIN_API purlin_status purlin_plan_device_error(purlin_plan_t plan, uint32_t* error);

/* Free a plan (NULL-safe).  Does not synchronise: the caller keeps the plan
 * alive until work queued with it has finished. */
PURLIN_API void purlin_plan_destroy(purlin_plan_t plan);

/* Whether purlin_pack runs in one launch for this shape (*single = 1) or in
 * three (*single = 0: per-tile metadata, its scan, then the rows).  The
 * one-launch form applies when every workgroup can count all T*K ids itself
 * and hold its tokens' rows in registers: rows a multiple of 16 bytes
 * (H % 8 == 0), 4 <= T*K <= 32768, E <= 1024, and at most 512 workgroups of
 * at most 64 tokens and 1024 (t, k) pairs each.  Both forms give the same
 * results (the definition below); the workspace is sized for either.
 * PURLIN_ERR_INVALID for NULL `single` or shapes purlin_pack rejects. */
PURLIN_API purlin_status purlin_pack_single_launch(int T, int H, int K, int E, int* single);

/* Workspace bytes purlin_pack needs for T tokens, K slots, E experts. */
PURLIN_API purlin_status purlin_pack_workspace_size(int T, int K, int E, uint64_t* bytes);

/* MoE dispatch (pack).  Expert parallelism dispatches tokens to the ranks
 * that own their experts (Section 2, Table 2); the variable-size segments
 * are the scatteredV layout of Section 3.1.  With L = E / P experts per
 * rank, expert e belongs to rank e / L, and
 *   expert_counts[e]  = #{(t,k) : ids[t,k] == e}
 *   expert_offsets[e] = sum of expert_counts[0..e)  (exclusive prefix sum)
 *   dest_counts[r]    = sum of expert_counts over rank r's experts
 *   dest_offsets[r]   = expert_offsets[r * L]
 *   pos[t,k]          = expert_offsets[e] + #{t' < t : e in ids[t',:]},  e = ids[t,k]
 *   packed[pos[t,k], :] = x[t, :]                              (bit copy)
 * so rows are grouped by destination rank, then expert, then token.
 *   x        bf16 [T, H] device, row-major
 *   ids      int32 [T, K] device; each id in [0, E), distinct within a token
 *   packed   bf16 [T*K, H] device (output)
 *   dest_counts, dest_offsets  int32 [P] device (output)
 *   expert_counts              int32 [E] device (output)
 *   expert_offsets             int32 [E] device (output, optional: NULL)
 *   pos      int32 [T, K] device (output)
 *   dev_status int32 device (optional: NULL): set to 0, or to 1 when an id
 *            is out of range or repeated within a token; then counts and
 *            positions are unspecified, pos holds -1 for out-of-range ids,
 *            and no row is written outside packed.
 *   workspace >= purlin_pack_workspace_size bytes of device memory, owned
 *            by the caller; its contents on entry do not matter.
 * Limits: T >= 0, H >= 1, 1 <= K <= 64, 1 <= E <= 4096, 1 <= P <= E,
 * E % P == 0, T*K < 2^31.  Errors: PURLIN_ERR_INVALID (limits, NULL or
 * misaligned pointer, small workspace), PURLIN_ERR_DEVICE. */
PURLIN_API purlin_status purlin_pack(int T, int H, int K, int E, int P, const void* x, const int32_t* ids,
                          void* packed, int32_t* dest_counts, int32_t* dest_offsets,
                          int32_t* expert_counts, int32_t* expert_offsets, int32_t* pos,
                          int32_t* dev_status, void* workspace, uint64_t workspace_bytes,
                          void* stream);

/* purlin_pack in two calls, so that the metadata, which reads only ids, can
 * run earlier or on another stream than the rows (Section 2, Table 2: the
 * dispatch; the counts are the scatteredV sizes of Section 3.1).
 * purlin_pack_meta computes dest_counts, dest_offsets, expert_counts,
 * expert_offsets and dev_status exactly as purlin_pack does, and leaves in
 * `workspace` what purlin_pack_rows needs; purlin_pack_rows then writes
 * packed and pos, bit-identical to purlin_pack.  Arguments have
 * purlin_pack's meaning and limits; the rows call must use the same T, K,
 * E and workspace, and must start after the metadata call has finished
 * (same stream, or an event between the streams); the workspace must not
 * be reused by another metadata call before the rows call has finished.
 * A rows call without a matching metadata call writes unspecified rows of
 * packed and pos, never outside them.  Errors: PURLIN_ERR_INVALID (limits,
 * NULL or misaligned pointer, small workspace, x overlapping packed),
 * PURLIN_ERR_DEVICE. */
PURLIN_API purlin_status purlin_pack_meta(int T, int K, int E, int P, const int32_t* ids, int32_t* dest_counts,
                                          int32_t* dest_offsets, int32_t* expert_counts, int32_t* expert_offsets,
                                          int32_t* dev_status, void* workspace, uint64_t workspace_bytes,
                                          void* stream);
PURLIN_API purlin_status purlin_pack_rows(int T, int H, int K, int E, const void* x, const int32_t* ids,
                                          void* packed, int32_t* pos, const void* workspace,
                                          uint64_t workspace_bytes, void* stream);

/* Bytes of the per-GPU workspace that purlin_pack_static uses instead of a
 * caller-supplied one. */
#define PURLIN_STATIC_SCRATCH_BYTES (4u << 20)

/* purlin_pack without the workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, outputs, bits
 * and errors as purlin_pack; the workspace is a library-owned array of
 * PURLIN_STATIC_SCRATCH_BYTES in device memory, one copy per GPU, held until
 * the process ends.  The call allocates nothing: on its first call on a
 * device (the current one, which `stream` must belong to) it looks that
 * copy's address up once.
 *   Limit: purlin_pack_workspace_size(T, K, E) <= PURLIN_STATIC_SCRATCH_BYTES
 *   (about 87 K tokens at K = 8, E = 256), else PURLIN_ERR_INVALID.
 *   Every call on one GPU shares its array: calls that may overlap on one
 *   GPU (different streams without ordering between them) race; order them
 *   on one stream.  PURLIN_ERR_UNSUPPORTED for a device index >= 64,
 *   PURLIN_ERR_DEVICE if the address lookup or a launch fails. */
PURLIN_API purlin_status purlin_pack_static(int T, int H, int K, int E, int P, const void* x, const int32_t* ids,
                                            void* packed, int32_t* dest_counts, int32_t* dest_offsets,
                                            int32_t* expert_counts, int32_t* expert_offsets, int32_t* pos,
                                            int32_t* dev_status, void* stream);

/* MoE combine (unpack), the inverse of purlin_pack weighted by gates:
 *   acc = +0.0f;
 *   for k = 0 .. K-1:  acc = acc + (gates[t,k] * widen(y[pos[t,k], h]));
 *   out[t, h] = narrow(acc)
 * each multiply and add a separately rounded binary32 operation (never
 * fused), slots summed in ascending order (the slot analogue of the rank
 * order of Eq. 2).
 *   y      bf16 [T*K, H] device (rows in purlin_pack's layout)
 *   pos    int32 [T, K] device, each in [0, T*K)
 *   gates  fp32 [T, K] device
 *   out    bf16 [T, H] device (output)
 *   dev_status int32 device (optional: NULL): set to 0, or to 1 if some pos
 *          is out of range (that slot then contributes nothing).
 * Limits: T >= 0, H >= 1, 1 <= K <= 64, T*K < 2^31.  Errors:
 * PURLIN_ERR_INVALID, PURLIN_ERR_DEVICE. */
PURLIN_API purlin_status purlin_unpack(int T, int H, int K, const void* y, const int32_t* pos,
                            const float* gates, void* out, int32_t* dev_status, void* stream);

/* Workspace bytes purlin_pack_dedup needs for T tokens over P ranks. */
PURLIN_API purlin_status purlin_pack_dedup_workspace_size(int T, int P, uint64_t* bytes);

/* De-duplicated MoE dispatch: one row per (token, destination rank) instead
 * of one per (token, slot).  A token whose K experts live on fewer than K
 * ranks is sent once to each of them (expert parallelism's dispatch, Section
 * 2, Table 2; the paper does not cover de-duplication, this is the
 * library's contract).  With L = E / P and dests(t) = {ids[t,k] / L}:
 *   dest_counts[r]  = #{t : r in dests(t)}
 *   dest_offsets[r] = sum of dest_counts[0..r)
 *   row_of[t, r]    = dest_offsets[r] + #{t' < t : r in dests(t')} if r in
 *                     dests(t), else -1
 *   packed[row_of[t, r], :] = x[t, :]                          (bit copy)
 * so rows are grouped by destination rank, then token.
 *   x        bf16 [T, H] device, row-major
 *   ids      int32 [T, K] device; each id in [0, E), distinct within a token
 *   packed   bf16 [T*min(K, P), H] device (output; the first
 *            sum(dest_counts) rows are written)
 *   dest_counts, dest_offsets  int32 [P] device (output)
 *   row_of   int32 [T, P] device (output)
 *   dev_status int32 device (optional: NULL): set to 0, or to 1 when an id
 *            is out of range or repeated within a token; out-of-range ids
 *            are then ignored, and no row is written outside packed.
 *   workspace >= purlin_pack_dedup_workspace_size bytes of device memory,
 *            owned by the caller; its contents on entry do not matter.
 * Limits: T >= 0, H >= 1, 1 <= K <= 64, 1 <= E <= 4096, 1 <= P <= 16,
 * P <= E, E % P == 0, T*K < 2^31.  Errors: PURLIN_ERR_INVALID (limits, NULL
 * or misaligned pointer, small workspace, x overlapping packed),
 * PURLIN_ERR_DEVICE. */
PURLIN_API purlin_status purlin_pack_dedup(int T, int H, int K, int E, int P, const void* x, const int32_t* ids,
                                           void* packed, int32_t* dest_counts, int32_t* dest_offsets,
                                           int32_t* row_of, int32_t* dev_status, void* workspace,
                                           uint64_t workspace_bytes, void* stream);

/* Combine of the de-duplicated dispatch: y holds one partial output per
 * (token, rank) in purlin_pack_dedup's layout (each rank has applied its
 * experts and their gates), and
 *   acc = +0.0f;
 *   for r = 0 .. P-1 with row_of[t, r] >= 0:  acc = acc + widen(y[row_of[t, r], h]);
 *   out[t, h] = narrow(acc)
 * binary32 adds in rank order (Eq. 2).
 *   y      bf16 [rows, H] device
 *   row_of int32 [T, P] device, each -1 or in [0, rows)
 *   out    bf16 [T, H] device (output)
 *   dev_status int32 device (optional: NULL): set to 0, or to 1 if some
 *          entry is neither -1 nor in [0, rows) (it then contributes
 *          nothing).
 * Limits: T >= 0, H >= 1, 1 <= P <= 16, 0 <= rows < 2^31.  Errors:
 * PURLIN_ERR_INVALID (limits, NULL or misaligned pointer, y overlapping
 * out), PURLIN_ERR_DEVICE. */
PURLIN_API purlin_status purlin_unpack_dedup(int T, int H, int P, int64_t rows, const void* y,
                                             const int32_t* row_of, void* out, int32_t* dev_status, void* stream);

/* Workspace bytes purlin_ep_dispatch needs for P ranks of T tokens. */
PURLIN_API purlin_status purlin_ep_dispatch_workspace_size(int T, int K, int E, int P, uint64_t* bytes);

/* Expert-parallel dispatch over P ranks in one pass (expert parallelism's
 * AllToAll(V) of tokens, Section 2, Table 2): the result is rank p's
 * purlin_pack followed by the ALLTOALLV of the packed rows with counts[p][r]
 * = rank p's dest_counts[r], but the rows go straight from x_p to the
 * receive buffers, with no packed buffers in between.  Rank r's buffer holds
 * the rows from rank 0, then rank 1, ..., each in its sender's pack order
 * (expert, then token).
 *   x        P host-held pointers to bf16 [T, H] device token rows
 *   ids      P host-held pointers to int32 [T, K] device expert ids
 *   recv     P host-held pointers to bf16 [capacity, H] device receive
 *            buffers (output; rows beyond what a rank receives untouched)
 *   counts   int32 [P * P] device (output): rows rank p sends rank r, at
 *            counts[p*P + r]
 *   recv_pos int32 [P, T, K] device (output): row of rank p's token t, slot
 *            k in the buffer of the rank owning expert ids_p[t, k]:
 *            sum_{q<p} counts[q][r] + pos_p[t,k] - dest_offsets_p[r]
 *   dev_status int32 device (optional): 0, or 1 if an id is out of range or
 *            repeated within a token (those slots are skipped), or if some
 *            rank would receive more than `capacity` rows (then no row is
 *            written).
 *   workspace >= purlin_ep_dispatch_workspace_size bytes of device memory,
 *            owned by the caller; its contents on entry do not matter.
 * Limits as purlin_pack, plus P <= 16, capacity < 2^31.  Errors:
 * PURLIN_ERR_INVALID (limits, NULL or misaligned pointer, small workspace,
 * a receive buffer overlapping another or a token buffer),
 * PURLIN_ERR_DEVICE. */
PURLIN_API purlin_status purlin_ep_dispatch(int T, int H, int K, int E, int P, const void* const* x,
                                            const int32_t* const* ids, void* const* recv, uint64_t capacity,
                                            int32_t* counts, int32_t* recv_pos, int32_t* dev_status,
                                            void* workspace, uint64_t workspace_bytes, void* stream);

/* The matching combine: the expert outputs y_r, in rank r's receive layout,
 * go back to their tokens and are summed in slot order as purlin_unpack
 * does:
 *   out_p[t, h] = narrow(+0 + g_p[t,0] * widen(y_{r0}[recv_pos[p,t,0], h]) + ...)
 * with r_k the rank owning ids_p[t, k] -- the same bits as the reverse
 * ALLTOALLV followed by purlin_unpack.
 *   y        P host-held pointers to bf16 [capacity, H] device
 *   ids, recv_pos  as given to / returned by purlin_ep_dispatch
 *   gates    P host-held pointers to fp32 [T, K] device
 *   out      P host-held pointers to bf16 [T, H] device (output)
 *   dev_status int32 device (optional): 0, or 1 if some slot names an id or
 *            a row out of range (it then contributes nothing).
 * Errors: PURLIN_ERR_INVALID (limits, NULL or misaligned pointer, an output
 * overlapping another or an input), PURLIN_ERR_DEVICE. */
PURLIN_API purlin_status purlin_ep_combine(int T, int H, int K, int E, int P, const void* const* y, uint64_t capacity,
                                           const int32_t* const* ids, const int32_t* recv_pos,
                                           const float* const* gates, void* const* out, int32_t* dev_status,
                                           void* stream);

/* Workspace bytes purlin_ep_dispatch_dedup needs for P ranks of T tokens. */
PURLIN_API purlin_status purlin_ep_dispatch_dedup_workspace_size(int T, int P, uint64_t* bytes);

/* The de-duplicated dispatch over P ranks in one pass: rank p's
 * purlin_pack_dedup followed by the ALLTOALLV of its rows, without the
 * packed buffers.  Rank r's buffer holds, from rank 0, then rank 1, ...,
 * one row per token having an expert on r, in token order.
 *   x, ids, recv, capacity, counts, dev_status, workspace  as
 *            purlin_ep_dispatch (counts[p*P + r] = tokens rank p sends r)
 *   recv_row int32 [P, T, P] device (output): row of rank p's token t in
 *            rank r's buffer, or -1 if none of its experts is on r:
 *            sum_{q<p} counts[q][r] + row_of_p[t,r] - dest_offsets_p[r]
 * Limits and errors as purlin_ep_dispatch. */
PURLIN_API purlin_status purlin_ep_dispatch_dedup(int T, int H, int K, int E, int P, const void* const* x,
                                                  const int32_t* const* ids, void* const* recv, uint64_t capacity,
                                                  int32_t* counts, int32_t* recv_row, int32_t* dev_status,
                                                  void* workspace, uint64_t workspace_bytes, void* stream);

/* Its combine: y_r holds rank r's partial outputs in its receive layout
 * (gates applied on the expert side), and
 *   out_p[t, h] = narrow(+0 + widen(y_r[recv_row[p,t,r], h]) for r = 0..P-1 with recv_row >= 0)
 * in rank order -- the same bits as the reverse ALLTOALLV followed by
 * purlin_unpack_dedup.  dev_status (optional): 0, or 1 if some entry is
 * neither -1 nor a row below `capacity` (it then contributes nothing).
 * Errors as purlin_ep_combine. */
PURLIN_API purlin_status purlin_ep_combine_dedup(int T, int H, int P, const void* const* y, uint64_t capacity,
                                                 const int32_t* recv_row, void* const* out, int32_t* dev_status,
                                                 void* stream);

/* Plain device-to-device copy of `bytes` bytes with no descriptors (each
 * lane moves 16-byte vectors; one 256-thread workgroup copies 16 KiB).  Not
 * a step of the method: it is the reference stream against which the
 * executor's copies are measured.
 *   dst, src  device pointers, 16-byte aligned, ranges disjoint
 *   bytes     a multiple of 16; 0 is a no-op
 * Asynchronous on `stream`.  PURLIN_ERR_INVALID: a null or misaligned
 * pointer (bytes > 0), bytes not a multiple of 16, overlapping ranges;
 * PURLIN_ERR_DEVICE: the launch failed. */
PURLIN_API purlin_status purlin_stream_copy(void* dst, const void* src, uint64_t bytes, void* stream);

/* Reference stream of n sources to m destinations with no descriptors:
 * for every 16-byte vector i < bytes / 16,
 *     v = src[0][i] ^ src[1][i] ^ ... ^ src[nsrc-1][i]   ({i, i, i, i} as
 *                                                        32-bit words if nsrc = 0)
 *     dst[j][i] = v  for every j < ndst
 * With ndst = 0 the sources are only read, and `sink` (16 bytes of device
 * memory) may receive an unspecified vector.  `hints`: PURLIN_STREAM_NT_LOAD
 * and / or PURLIN_STREAM_NT_STORE select non-temporal loads / stores.  Not a step of the method:
 * the streams (read-only, write-only, 1:1, 8-to-1, 1-to-8) are the access
 * mixes the executor's kernels are measured against.
 *   dst   ndst device pointers, 16-byte aligned, pairwise disjoint ranges
 *   src   nsrc device pointers, 16-byte aligned (may alias each other)
 *   bytes a multiple of 16; 0 is a no-op
 * 0 <= nsrc, ndst <= 16, nsrc + ndst >= 1.  Asynchronous on `stream`.
 * PURLIN_ERR_INVALID: counts out of range, bytes not a multiple of 16, a
 * NULL or misaligned pointer, a destination overlapping a source or
 * another destination, ndst = 0 without a sink, unknown hint bits;
 * PURLIN_ERR_DEVICE: the launch failed. */
#define PURLIN_STREAM_NT_LOAD 1u
#define PURLIN_STREAM_NT_STORE 2u
PURLIN_API purlin_status purlin_stream(void* const* dst, int ndst, const void* const* src, int nsrc, uint64_t bytes,
                                       void* sink, uint32_t hints, void* stream);

/* Measurement entry points: purlin_stream and the one-launch purlin_pack,
 * each also recording when every workgroup ran and on which XCD (the
 * chip's accelerator dies, which the hardware deals consecutive workgroups
 * to round-robin), so that a kernel's time can be split into its dies'
 * finishing times.  Not
 * steps of the method.  `rec` (device, 16-byte aligned, rec_entries
 * uint64 entries, at least 4 * (groups + 1)) receives
 *   rec[0] = the wall-clock rate in kHz, rec[1] = groups,
 *   rec[4(b+1) + 0..3] = {XCD id, wall clock at entry, wall clock when the
 *                        workgroup's metadata was done (its entry for a
 *                        stream), wall clock once all its stores completed}
 * for every workgroup b.  The recording adds one wait and one barrier at the
 * end of each workgroup.  `groups` (host, optional) receives the number of
 * workgroups; with rec = NULL nothing is launched (a size query).
 * purlin_stream_timed: arguments and errors as purlin_stream, plus
 * PURLIN_ERR_INVALID for a short, misaligned or overlapping rec.
 * purlin_pack_timed: arguments, results and errors as purlin_pack (no
 * workspace), for shapes purlin_pack_single_launch accepts; other shapes
 * give PURLIN_ERR_UNSUPPORTED. */
PURLIN_API purlin_status purlin_stream_timed(void* const* dst, int ndst, const void* const* src, int nsrc,
                                             uint64_t bytes, void* sink, uint32_t hints, uint64_t* rec,
                                             uint64_t rec_entries, uint64_t* groups, void* stream);
PURLIN_API purlin_status purlin_pack_timed(int T, int H, int K, int E, int P, const void* x, const int32_t* ids,
                                           void* packed, int32_t* dest_counts, int32_t* dest_offsets,
                                           int32_t* expert_counts, int32_t* expert_offsets, int32_t* pos,
                                           int32_t* dev_status, uint64_t* rec, uint64_t rec_entries,
                                           uint64_t* groups, void* stream);

/* Static text for a status code ("unknown status" for others). */
PURLIN_API const char* purlin_status_string(purlin_status status);

/* Library version, e.g. "0.1.0" (static text). */
PURLIN_API const char* purlin_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PURLIN_H */
