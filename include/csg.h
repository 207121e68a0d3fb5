/*
 * csg.h -- chunk-scheduled GEMM for MI355X (gfx950): the C ABI.
 *
 * One persistent GEMM kernel whose tile scheduler follows a communication-chunk
 * schedule (Syncopate, arXiv 2601.20595, Section 5.2): tiles that consume a
 * chunk wait for that chunk's ready flag and are visited in chunk-arrival
 * order; tiles that produce an output chunk signal it when the chunk is
 * complete. On one GPU the "remote" side of a rank is simulated: remote shards
 * are staged in HBM and moved by SDMA copy-engine copies (Section 2.3, copy
 * engine backend; Section 5.2, realization (1): copy engine + global-memory
 * signals). Copies are issued by the calling thread straight to the SDMA engines.
 * Overlap GEMM calls and every copy-only call return once their copies are issued (an
 * overlap kernel waits for each chunk's copy; csg_plan_check waits for all of them,
 * and csg_plan_join makes a stream wait for them on the device); ring-attention
 * overlap calls return once their copies have completed. Either way the kernel may
 * still be running on the compute stream.
 *
 * Conventions for every entry point
 *   - Every call returns csg_status; nothing throws or aborts across the ABI.
 *     A failing call leaves a thread-local message readable by csg_last_error().
 *   - Ordering against the caller's streams: a call's kernels follow the work already
 *     queued on its compute stream, and its copies the work already queued on its
 *     copy stream. Inputs written on any other stream (the default one included) must
 *     be complete before the call.
 *   - Pointers named *_host are host memory; every other data pointer is device
 *     memory of the plan's device, owned by the caller. Streams are hipStream_t
 *     values passed as void*; they are owned by the caller and must belong to
 *     the plan's device.
 *   - Matrices are dense row-major with no padding: A is M x K, B is N x K
 *     (K contiguous, the local kernel's a . b^T form), C is M x N; grouped
 *     weights are E x N x K. dtype CSG_BF16 elements are raw bfloat16 bit
 *     patterns (uint16), CSG_F32 are IEEE binary32.
 *   - Objects (schedules, plans) are not thread-safe; distinct objects are
 *     independent. The kernels of one plan run in call order: the plan's per-call
 *     state is reset, and its copies wait for earlier readers, in that order. Pass
 *     the same compute stream to successive calls; a call on another stream first
 *     makes that stream wait for the previous call's kernel and prologue.
 */
#ifndef CSG_H_
#define CSG_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CSG_OK = 0,
    CSG_ERR_INVALID = 1,      /* bad argument or schedule; nothing was enqueued */
    CSG_ERR_UNSUPPORTED = 2,  /* valid request this build cannot serve (device, dtype, tile) */
    CSG_ERR_HIP = 3,          /* a HIP runtime call failed; csg_last_error() has its text */
    CSG_ERR_NOMEM = 4,        /* host or device allocation failed */
    CSG_ERR_TIMEOUT = 5,      /* a bounded wait expired (see csg_diag) */
    CSG_ERR_STATE = 6         /* call not allowed in the object's current state */
} csg_status;

typedef enum { CSG_BF16 = 0, CSG_F32 = 1 } csg_dtype;

typedef enum {
    CSG_AG_GEMM = 0,        /* AllGather(A) + GEMM: tiles consume arriving A row chunks */
    CSG_GEMM_RS = 1,        /* GEMM + ReduceScatter: tiles produce C row chunks that are sent */
    CSG_GROUPED_GEMM = 2,   /* all-to-all(X) + grouped GEMM: per-(source, expert) row segments */
    CSG_GEMM_AR = 3         /* GEMM + AllReduce (reduce-scatter then all-gather of C row chunks) */
} csg_op;

typedef enum {
    CSG_ORDER_RING = 0,         /* local shard, then shards r-1, r-2, ... (ring AllGather) */
    CSG_ORDER_SWIZZLE1D = 1,    /* local shard, then peers (i + r) mod W, i = 1..W-1 */
    CSG_ORDER_PERMUTATION = 2,  /* local chunks, then remote chunks in a caller-given order */
    CSG_ORDER_RS_RING = 3       /* shards (r + 1 + t) mod W, t = 0..W-1 (own shard last) */
} csg_order;

/* What moves the chunks (Section 5.2, communication code generation: the same
 * chunk schedule realised by different mechanisms). */
typedef enum {
    CSG_COPY_SDMA = 0,    /* copy engines, driven by the calling thread, with completion
                             signals as the chunks' ready flags (realization (1)) */
    CSG_COPY_KERNEL = 1   /* the GEMM kernel's own workgroups, by vector loads and stores:
                             AG / grouped: workgroups 0 .. copy_workgroups - 1 (the first
                             the device starts) move the remote chunks in arrival order,
                             raise each chunk's ready flag, then take tiles (realization
                             (4), specialised workgroups); GEMM-RS: a tile of a chunk that is sent also
                             stores its output rows into the outgoing buffer from its
                             epilogue (realization (5), co-located), which needs every
                             chunk to start on a multiple of bm */
} csg_copy_backend;

typedef enum {
    CSG_MODE_OVERLAP = 0,       /* copies and kernel run concurrently */
    CSG_MODE_COMPUTE_ONLY = 1,  /* every flag pre-set, no copies; the kernel still polls */
    CSG_MODE_COPY_ONLY = 2      /* copies only (reduce-scatter: C must already hold the output) */
} csg_mode;

/* One chunk: the contiguous row range [row_begin, row_end) of A (AG, grouped) or
 * of C (RS) moved as one unit (Section 5.1, chunk definition). src_rank is the
 * rank that owns it, group the expert index (grouped GEMM; 0 otherwise),
 * is_local != 0 when the chunk is already on this rank (never copied). */
typedef struct {
    int64_t row_begin;
    int64_t row_end;
    int32_t src_rank;
    int32_t group;
    int32_t is_local;
    int32_t reserved;       /* must be 0 */
} csg_chunk;

/* Tile and runtime knobs. Zero means "default" for every field.
 *   bm, bn, bk      tile shape; must name a compiled kernel variant on a device plan
 *                   (bk = 64 for bf16, 16 for fp32): bf16 inputs 256 x 256 (every operation;
 *                   the default), 256 x 224 (all-gather and grouped GEMMs), 128 x 256
 *                   (those and GEMM + reduce-scatter, bf16 output), 256 x 128 and 128 x 128
 *                   (all-gather and grouped GEMMs, bf16 output); fp32 inputs 64 x 64
 *   intra_order     tile order inside a chunk (Section 5.2, intra-chunk swizzle), the
 *                   chunk order staying as it is: 0 = raster (m, n), the local kernel's
 *                   own traversal; 1 = the row tiles sharing a chunk key, ascending, are
 *                   cut into bands of group_m and each band is visited column by column:
 *                   order = (key, band, n, m)
 *   group_m         band height of intra_order 1 (0 = 8)
 *   tile_dispatch   0 or 1 = workgroups take the next entry of the tile list from an
 *                   atomic ticket; 2 = static: workgroup w takes entries s, s + G, s + 2G,
 *                   ... with s = (w mod 8) * (G / 8) + w / 8 when G is a multiple of 8
 *                   (else s = w), so that the workgroups of one die (the dispatcher
 *                   deals workgroups to the 8 dies round robin) take consecutive entries;
 *                   with a tail split (all-gather and grouped GEMMs) the units of the
 *                   split tail tiles, which end the list, are taken in order from a
 *                   shared ticket by whichever workgroup is free first
 *   num_workgroups  persistent grid size G (0 = one per co-resident slot)
 *   copy_engines    SDMA engines the chunk copies are spread over (0 = every engine the
 *                   device offers for device-to-device copies)
 *   timeout_ms      bound on every wait (kernel flag polls, host waits); 0 = 2000
 *   split_k         K-slices per tile (0 or 1 = none): the slices of a tile run on different
 *                   workgroups and the last one to finish adds the fp32 partial sums in slice
 *                   order, so the result depends on split_k but not on timing; a larger value
 *                   shortens the work left after the last chunk lands (and the first emission)
 *   tail_split      K-slices for the tiles on the overlap's critical path: the tiles that
 *   tail_chunks     read one of the tail_chunks last-arriving chunks (AG, grouped) or write
 *                   one of the tail_chunks first-emitted chunks (RS); 0 = none. Slices are
 *                   added as for split_k (the slices exchange fp32 partial sums through
 *                   memory, so they may run on any die). A plan with split tiles of
 *                   either kind takes a num_workgroups, if given, that is a multiple of 8
 *   trace           1 = the kernel records when each work unit was taken, started and
 *                   finished (read back with csg_plan_trace); 0 = off
 *   warm_rows       consumers: 0 or 1 = a workgroup that sees a chunk land first loads
 *                   its share of the tile's A rows into the caches before computing
 *                   (copy-engine writes leave the rows only in HBM); 2 = off
 *   copy_backend    a csg_copy_backend value; 0 = CSG_COPY_SDMA
 *   copy_workgroups CSG_COPY_KERNEL: workgroups that move chunks (0 = 16); a copy-only
 *                   call launches exactly this many
 *   tail_wave       > 1: each die's tile list ends in a partial wave of L mod w tiles (w =
 *                   the die's workgroups), which would run with the rest of the die idle;
 *                   those tiles are split into min(tail_wave, w / (L mod w)) K-slices
 *                   (added as for split_k). Per-die dispatch only (tile_dispatch 0/1);
 *                   0 or 1 = off
 *   copy_split      copy engines, all-gather, grouped and reduce-scatter plans: > 1 = a
 *                   chunk copy may be cut into up to copy_split pieces (of at least
 *                   512 KiB), each on its own engine. The library models each engine's
 *                   queue (about 48 GB/s per engine) and gives a copy the engines
 *                   expected to be free first, in the number of pieces that lands it
 *                   soonest: copies issued while the engines are busy stay whole, a copy
 *                   issued to idle engines lands in a fraction of one engine's time.
 *                   The chunk's signal is armed to 1 and raised by pieces - 1 before the
 *                   pieces are issued; each piece brings it down by one. 0 or 1 = every
 *                   chunk whole, on engine (i mod engines) for the i-th copy
 *   tail_taper      1 = the tail split tapers: the tiles of the j-th of the tail_chunks
 *                   chunks, counted from the last to arrive (AG, grouped) or the first
 *                   emitted (RS), get ceil(S / (1 + j (S - 1) / (C - 1))) K-slices, S =
 *                   tail_split, C = tail_chunks (S for the last chunk, 1 for the C-th);
 *                   0 = every tail tile gets tail_split slices */
typedef struct {
    int32_t bm, bn, bk;
    int32_t intra_order;
    int32_t tile_dispatch;
    int32_t num_workgroups;
    int32_t copy_engines;
    int32_t timeout_ms;
    int32_t split_k;
    int32_t tail_split;
    int32_t tail_chunks;
    int32_t trace;
    int32_t warm_rows;
    int32_t copy_backend;
    int32_t copy_workgroups;
    int32_t group_m;
    int32_t tail_wave;
    int32_t copy_split;
    int32_t tail_taper;
} csg_plan_cfg;

typedef struct csg_schedule csg_schedule;
typedef struct csg_plan csg_plan;

typedef struct {
    int32_t n_tiles;        /* tiles of the output */
    int32_t n_chunks;
    int32_t nnz;            /* sum over tiles of the chunks each tile touches */
    int32_t n_tiles_n;      /* tiles along N */
    int32_t num_workgroups; /* persistent grid actually used (0 on a host-only plan) */
    int32_t bm, bn, bk;     /* tile shape actually used */
    int32_t n_units;        /* work units of the execution list (0 on a host-only plan) */
} csg_plan_info;

/* One work unit (a tile, or one K-slice of a split tile) of the last kernel run of a
 * plan with tracing on, in execution-list order. Times are device wall-clock ticks
 * (100 MHz): when a workgroup took the unit, when the unit's chunk waits were over,
 * and when the unit finished (its output stored, or its partial sums for a slice
 * that was not the last), and the shader-clock cycles in between, so that
 * cycles / (t_end - t_start) * 100 MHz is the clock the unit ran at. */
typedef struct {
    int32_t raster;         /* raster id of the tile */
    int32_t slice;          /* K-slice index */
    int32_t n_slices;       /* K-slices of the tile (1 = not split) */
    int32_t xcd;            /* die the workgroup ran on */
    int32_t workgroup;      /* workgroup id */
    int32_t reserved;
    uint64_t t_take, t_start, t_end;
    uint64_t cycles;        /* shader-clock cycles from t_start to t_end */
} csg_trace_unit;

/* Diagnostics of the last call on a plan (filled by csg_plan_check). */
typedef struct {
    int32_t timed_out;      /* 1 if a kernel flag wait or a host wait expired */
    int32_t chunk;          /* chunk id waited on, -1 if none */
    int32_t tile;           /* raster id of the tile that waited, -1 if none */
    uint32_t observed;      /* value seen when the wait gave up (the chunk copy's completion
                               signal: 1 = not landed) */
    uint32_t epoch;         /* call number of the plan */
    int32_t reserved;
} csg_diag;

/* Library version string, static storage. */
const char* csg_version(void);

/* Human-readable name of a status, static storage. */
const char* csg_status_str(csg_status s);

/* Message of the last failing call on this thread ("" if none), thread-local storage. */
const char* csg_last_error(void);

/* Writes the device's architecture name into arch (NUL-terminated, truncated to
 * arch_len). CSG_OK if it is gfx950, CSG_ERR_UNSUPPORTED otherwise, CSG_ERR_HIP if
 * the device cannot be queried. */
csg_status csg_device_check(int device, char* arch, size_t arch_len);

/* ---- schedules (host only; Section 5.1) ---------------------------------------- */

/* General schedule: n chunks (copied) that must tile [0, chunks[n-1].row_end) in
 * row order, each non-empty, and order[0..n-1] a permutation of 0..n-1 giving the
 * arrival (AG, grouped) or emission (RS) order. CSG_ERR_INVALID otherwise. */
csg_status csg_schedule_create(const csg_chunk* chunks, int32_t n, const int32_t* order,
                               csg_schedule** out);

/* Uniform schedule of one rank (template specialisation, Section 5.1): world
 * ranks each own shard_rows rows split into chunks_per_shard equal chunks; chunk
 * c = s*Q + q covers rows [s*S + q*h, s*S + (q+1)*h). For CSG_ORDER_PERMUTATION,
 * remote_perm_host holds a permutation of 0..(world-1)*Q-1 applied to the
 * ascending list of remote chunk ids (it is ignored, and may be NULL, for the
 * other orders). */
csg_status csg_schedule_uniform(int32_t world, int32_t rank, int64_t shard_rows,
                                int32_t chunks_per_shard, csg_order order,
                                const int32_t* remote_perm_host, csg_schedule** out);

/* All-to-all schedule of one rank: counts_host[s * n_groups + e] routed rows come
 * from source rank s for local expert e. Rows are laid out expert-major, then
 * source-major; each non-empty (s, e) segment is a chunk of group e; arrival is
 * the rank's own segments, then sources r-1, r-2, ..., experts ascending. */
csg_status csg_schedule_grouped(int32_t world, int32_t rank, int32_t n_groups,
                                const int64_t* counts_host, csg_schedule** out);

/* Number of chunks and rows covered. */
csg_status csg_schedule_info(const csg_schedule* s, int32_t* n_chunks, int64_t* total_rows);

/* Copies the chunk list and the order out (arrays of n_chunks entries; either may be NULL). */
csg_status csg_schedule_get(const csg_schedule* s, csg_chunk* chunks_host, int32_t* order_host);

void csg_schedule_destroy(csg_schedule* s);

/* ---- plans ------------------------------------------------------------------ */

/* Builds the chunk-tile dependence map and the chunk-ordered tile list
 * (Section 5.2: dependency parsing, tile-scheduler swizzling) for
 * C[M x N] = A[M x K] . B[N x K]^T under schedule s, and, when device >= 0, the
 * device state one call needs (tile list, wait lists, flags, counters).
 * device < 0 makes a host-only plan: the map can be read, no GEMM can run.
 * op CSG_GROUPED_GEMM needs group_rows_host[n_groups] (rows per expert, summing to
 * M) and chunks that stay inside their group; other ops pass NULL, 0.
 * The schedule is copied; it may be destroyed afterwards.
 * CSG_ERR_INVALID for a malformed request (M not the rows the chunks cover, a bad
 * configuration field); CSG_ERR_UNSUPPORTED, for host-only plans too, when K is not a
 * multiple of the main loop's K step (cfg bk: 64 for bf16, 16 for fp32), N is not a
 * multiple of 4, or there are more than 4096 chunks; on a device also when no kernel
 * variant has the tile shape, or a tile's rows exceed 32-bit buffer offsets. */
csg_status csg_plan_create(csg_op op, int64_t M, int64_t N, int64_t K, csg_dtype in_dtype,
                           csg_dtype out_dtype, const csg_schedule* s,
                           const int64_t* group_rows_host, int32_t n_groups,
                           const csg_plan_cfg* cfg, int device, csg_plan** out);

csg_status csg_plan_info_get(const csg_plan* p, csg_plan_info* info);

/* Copies out the map, all host arrays (any may be NULL):
 *   tile_ptr[n_tiles+1], tile_chunks[nnz]   D(t): ascending chunk ids per raster tile id
 *   chunk_ptr[n_chunks+1], chunk_tiles[nnz] T(c): ascending raster tile ids per chunk
 *   tile_order[n_tiles]                     raster ids in execution order, sorted by
 *                                           (max (consumers) / min (RS) arrival position
 *                                           of D(t), raster id)
 * Raster id = global row-tile index * n_tiles_n + n; grouped row tiles are numbered
 * group by group. */
csg_status csg_plan_get_map(const csg_plan* p, int32_t* tile_ptr, int32_t* tile_chunks,
                            int32_t* chunk_ptr, int32_t* chunk_tiles, int32_t* tile_order);

/* Per-remote-chunk release delays in microseconds, in arrival order
 * (n = number of remote chunks); the chunk at arrival position i of the remote
 * chunks is not copied before sum_{j<=i} delay_us[j] after the call starts.
 * NULL clears them. With delays set, copies are issued from the calling thread
 * at their release times, so the call returns only after the last copy is
 * issued. With CSG_COPY_KERNEL the copy workgroups wait for the release times
 * instead, counted from when the call's prologue runs on the device; setting
 * delays then waits for the plan's kernels to finish. */
csg_status csg_plan_set_copy_delays(csg_plan* p, const float* delay_us_host, int32_t n);

/* AllGather + GEMM on one rank. a_landing is the full M x K A whose local rows are
 * already in place; a_staging has the same layout and holds the remote rows (the
 * simulated peers' shards). The prologue and the persistent kernel are queued on
 * `compute`; then, once the work queued earlier on `copy` has completed, the
 * calling thread issues, for each remote chunk in arrival order, an SDMA copy
 * staging -> landing whose completion signal is the chunk's ready flag. Before a
 * copy overwrites landing rows it waits for the plan's earlier kernels that read
 * them: after a call on the same a_landing, until that call's kernel has read the
 * chunk; after a call on a different buffer that overlaps it, until that kernel has
 * read every chunk; a buffer no earlier call of the plan overlaps (say, the other
 * of two activations used in turn) needs no wait. In overlap mode the call returns
 * once every copy is issued (the kernel waits for each, and csg_plan_check for
 * all); so does copy-only mode (csg_plan_check or csg_plan_join wait for the
 * copies). The kernel runs
 * tiles in chunk order, each waiting for its chunks. Work queued on `compute`
 * afterwards is ordered after the kernel. Asynchronous failures (a flag wait that
 * timed out) surface through csg_plan_check. CSG_ERR_TIMEOUT if a host wait
 * expired.
 * With CSG_COPY_KERNEL the call only queues the prologue and the kernel on
 * `compute` (its copy workgroups move the chunks; copy-only: they alone run) and
 * returns; `copy` is not used. */
csg_status csg_ag_gemm(csg_plan* p, void* a_landing, const void* a_staging, const void* b_nk,
                       void* c, csg_mode mode, void* compute_stream, void* copy_stream);

/* For callers that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc. The all-gather GEMM of csg_ag_gemm with
 * the chunks moved by the kernel's own copy workgroups (as with
 * csg_plan_cfg.copy_backend = CSG_COPY_KERNEL; no copy engine, no signal), without a
 * plan: every table it needs (work units, chunk lists, copy slabs) and every per-call
 * word (tickets, counters, ready words, diagnostics) lives in a static device array of
 * the library, 2 MiB per device, which each device the library runs on holds from the
 * library's load until the process ends. The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); it queues a table upload when the schedule,
 * shape or dtypes differ from the previous call's on the device, then a prologue and
 * the kernel, all on `stream` (a hipStream_t of `device`), and returns.
 * Arguments as for csg_plan_create + csg_ag_gemm: `s` (host; not kept after the call)
 * covers exactly M rows; a_landing (M x K, local rows in place), a_staging (same
 * layout, the remote rows), b_nk (N x K), c (M x N) are device buffers of `device`,
 * 16-byte aligned; tiles are 256 x 256 x 64 (bf16 input) or 64 x 64 x 16 (f32), dispatched
 * per die with stealing, not split. copy_workgroups: workgroups that move the chunks
 * (0 = 16). Modes as for csg_ag_gemm (compute-only: a_landing already holds every row;
 * copy-only: the copy workgroups alone run).
 * Limits: at most 4096 chunks, 16384 tiles, 32768 (tile, remote chunk) pairs and 16384
 * copy slabs of 256 KiB (4 GiB of remote rows); beyond them CSG_ERR_UNSUPPORTED, before
 * anything is queued. Every other check of csg_plan_create and csg_ag_gemm applies
 * (CSG_ERR_INVALID / CSG_ERR_UNSUPPORTED).
 * All calls on one device share its array, which keeps the last call's tables: calls
 * that may overlap on one device (on different streams, or from several threads without
 * an order between their streams) race and give wrong results; calls queued on one
 * stream are ordered. A flag wait that times out (2 s; the kernel's own copy workgroups
 * move every chunk, so only a stalled device gets there) is not reported. */
csg_status csg_ag_gemm_noalloc(const csg_schedule* s, int64_t M, int64_t N, int64_t K, csg_dtype in_dtype,
                               csg_dtype out_dtype, void* a_landing, const void* a_staging, const void* b_nk,
                               void* c, csg_mode mode, int32_t copy_workgroups, int device, void* stream);

/* GEMM + ReduceScatter on one rank: the kernel computes C tiles in emission
 * order; the last tile of an output chunk releases the chunk's flag, and the
 * calling thread then copies the chunk by SDMA from c to c_outgoing (non-local
 * chunks only). The call returns once the kernel has emitted its last non-local
 * chunk and every copy has been issued; the copies complete on their own. The next
 * call's kernel waits for the copy out of a chunk before rewriting its rows of c, and
 * csg_plan_check waits for all of them: call it (or csg_plan_destroy) before reading
 * c_outgoing. In copy-only mode c must already hold the output (the plan's previous
 * kernel is waited for).
 * With CSG_COPY_KERNEL the call only queues the prologue and the kernel on
 * `compute` and returns; `copy` is not used. Overlap: the tiles of a non-local chunk
 * store their output rows into both c and c_outgoing, and the chunk is sent when its
 * last tile has stored; copy-only: copy workgroups move the non-local chunks' rows
 * c -> c_outgoing, after the work queued earlier on `compute`. */
csg_status csg_gemm_rs(csg_plan* p, const void* a, const void* b_nk, void* c, void* c_outgoing,
                       csg_mode mode, void* compute_stream, void* copy_stream);

/* GEMM + AllReduce on one rank (Evaluation, the GEMM-AR operator; Section 5.1, the
 * partition-based AllReduce schedule), as a reduce-scatter then an all-gather of C row
 * chunks. Every rank holds a K-slice of a row-parallel product; the result is the sum
 * of all ranks' partial products a . b_nk^T. The plan's schedule is that of
 * GEMM-RS (emission order, own shard last; every chunk the same height; the local
 * chunks, contiguous, are the own shard of S rows, starting and ending on tile rows;
 * M = world * S). The kernel computes this rank's partial in emission order:
 *   - a non-local chunk's partial rows go to c; once emitted, the calling thread sends
 *     them by SDMA (c -> c_outgoing) and then copies that chunk's all-reduced rows,
 *     which its owner sends (reduced_staging, M x N, same row offsets), into the same
 *     rows of c, on the same engine after the send;
 *   - a tile of the own shard first waits for the other ranks' partial sums of its rows
 *     (partials_staging -> partials_landing by SDMA, [world-1][S][N] in C's element
 *     type, ranks in ascending order without this one, copied at the start of the
 *     call), adds them to its fp32 accumulators in that order, and stores the reduced
 *     rows; each reduced own chunk is then sent (c -> c_outgoing).
 * When every copy is done, c holds the all-reduced M x N result and c_outgoing what
 * this rank sent. The call returns once every copy has been issued; the copies
 * complete on their own (the next call's kernel waits per chunk for the last copy of
 * its rows; csg_plan_check waits for all). Compute-only: partials_landing must already
 * hold the partials, nothing is copied (c's non-local rows keep the partial products).
 * Copy-only: the copies alone, on what c holds (the previous kernel is waited for).
 * CSG_ERR_UNSUPPORTED at plan creation for schedules not of that form, split tiles or
 * the kernel copy backend. */
csg_status csg_gemm_ar(csg_plan* p, const void* a, const void* b_nk, void* c, void* c_outgoing,
                       const void* partials_staging, void* partials_landing,
                       const void* reduced_staging, csg_mode mode, void* compute_stream,
                       void* copy_stream);

/* All-to-all + grouped GEMM on one rank: x_landing / x_staging as in csg_ag_gemm
 * (expert-major rows), b_enk the E x N x K expert weights; tile rows never cross
 * an expert boundary. */
csg_status csg_grouped_gemm(csg_plan* p, void* x_landing, const void* x_staging,
                            const void* b_enk, void* c, csg_mode mode, void* compute_stream,
                            void* copy_stream);

/* ---- ring attention (Evaluation, the Ring-Attn operator; Section 5.2) ------------- */

/* Sequence-parallel attention on one rank: the rank's q_rows queries (n_heads heads
 * of head_dim) attend to every rank's keys and values, whose rows arrive in chunks
 * by the schedule kv_schedule (chunks over key rows, arrival order; local chunks
 * are the rank's own keys). Key/value heads are shared by n_heads / n_kv_heads
 * query heads each. The kernel supports head_dim 128 (else CSG_ERR_UNSUPPORTED) and
 * chunks of a multiple of 64 key rows; cfg may set timeout_ms, copy_engines and
 * num_workgroups (others must be 0). Free with csg_plan_destroy; csg_plan_check and
 * csg_plan_kernel_times apply. */
csg_status csg_attn_plan_create(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                int64_t q_rows, const csg_schedule* kv_schedule,
                                const csg_plan_cfg* cfg, int device, csg_plan** out);

/* One ring-attention call. Layouts (bf16, row-major, no padding): q and o are
 * [q_rows][n_heads][head_dim]; k_landing / v_landing (and k_staging / v_staging, the
 * simulated peers' shards at the same offsets) are [S][n_kv_heads][head_dim] with S
 * the schedule's key rows, the local rows already in place in the landing buffers;
 * lse is float [n_heads][q_rows], the natural-log log-sum-exp of each row's scaled
 * scores. The result, for every query row and head, is softmax(q . k^T / sqrt(d)) . v
 * over all S keys (no mask). As for csg_ag_gemm: the kernel is queued on `compute`,
 * the calling thread copies each remote chunk's keys and values by SDMA (two copies,
 * one completion signal as the chunk's ready flag) once the previous call's kernel
 * has finished reading those rows, and returns when the copies have completed
 * (copy-only mode: once they are issued, as for csg_ag_gemm). Each
 * work unit (one head, 128 query rows) consumes the chunks in arrival order, waiting
 * for each once. Compute-only: the landing buffers must already hold every row. */
csg_status csg_ring_attn(csg_plan* p, const void* q, void* k_landing, void* v_landing,
                         const void* k_staging, const void* v_staging, void* o, void* lse,
                         csg_mode mode, void* compute_stream, void* copy_stream);

/* Waits for the plan's last call to complete (its kernel and every copy it issued)
 * and reports its diagnostics.
 * CSG_ERR_TIMEOUT if a wait expired (details in *out); CSG_ERR_STATE if the kernel
 * finished without running every work unit (which only a grid that leaves a die
 * without workgroups can cause); CSG_OK otherwise. */
csg_status csg_plan_check(csg_plan* p, csg_diag* out);

/* Makes `stream` (a hipStream_t of the plan's device) wait, on the device, until every
 * copy the plan's last call issued has completed: a one-workgroup kernel is queued on
 * it whose threads poll the copies' completion signals (one thread per signal, up to
 * 256 at a time), at most the plan's timeout_ms per copy
 * (a copy still running then is reported by csg_plan_check, not here). Work queued on
 * `stream` afterwards follows the copies without a host wait, e.g. a consumer of
 * GEMM-RS's outgoing buffer, or an event that timestamps the end of the call's copies.
 * Queued on the call's compute stream it also follows the call's kernel. Enqueues
 * nothing for plans whose kernel moves the chunks itself (CSG_COPY_KERNEL: the kernel
 * covers its copies) or that never ran. CSG_ERR_STATE on a host-only plan. */
csg_status csg_plan_join(csg_plan* p, void* stream);

/* MFMA microbenchmark (a measurement aid, not part of any call above): one workgroup
 * of four waves per CU of `device`, each wave issuing `iters` rounds of 8 independent
 * bf16 32x32x16 MFMAs on register operands. *tflops receives the dense bf16 rate the
 * device sustained (2 * 32 * 32 * 16 flops per MFMA over the dispatch's own start and
 * end timestamps), *ms (may be NULL) the kernel's duration and *ghz (may be NULL) the
 * shader clock of workgroup 0 over its loop. The rate falls with the clock as a longer
 * run heats the device, so the measured peak depends on iters (about 1 ms per 7800
 * iterations at 2 GHz). Allocates and frees its own small buffers; synchronous.
 * CSG_ERR_UNSUPPORTED unless the device is gfx950. */
csg_status csg_measure_mfma_peak(int device, int32_t iters, double* tflops, double* ms, double* ghz);

/* Durations of the plan's most recent GEMM kernel launches, oldest first: the time
 * between two timing events the library records on the compute stream right
 * before and right after each kernel (so it covers the kernel only, not the
 * prologue or host launch latency; in overlap mode it includes the kernel's
 * waits for chunks). Up to n values (at most the last 256 launches) are written to
 * ms_host; *n_out receives how many. Waits for those launches to complete.
 * CSG_ERR_STATE on a host-only plan, CSG_ERR_INVALID for n < 0 or NULL
 * pointers. */
csg_status csg_plan_kernel_times(csg_plan* p, float* ms_host, int32_t n, int32_t* n_out);

/* Copies the trace of the plan's last kernel run (plan created with cfg.trace = 1)
 * into units_host[0..n): at most n units, *n_out receives how many. Waits for the
 * kernel. CSG_ERR_STATE if the plan does not trace or never ran a kernel,
 * CSG_ERR_INVALID for NULL pointers or n < 0. */
csg_status csg_plan_trace(csg_plan* p, csg_trace_unit* units_host, int32_t n, int32_t* n_out);

/* Waits for the plan's last call, then frees everything the plan owns. */
void csg_plan_destroy(csg_plan* p);

#ifdef __cplusplus
}
#endif

#endif /* CSG_H_ */
