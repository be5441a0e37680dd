/*
 * reshard.h -- C ABI of libreshard.so: cross-mesh resharding on one MI355X.
 *
 * Problem (Zhuang et al., "On Optimizing the Communication of Model
 * Parallelism", MLSys 2023, Section 2.2 "Cross-mesh resharding"): a tensor D
 * laid out on a source device mesh under sharding spec X_A must be laid out
 * on a disjoint destination mesh under spec X_B.  The library decomposes the
 * task into unit communication tasks (one per unique data slice, Section 2.2
 * and the appendix decomposition), picks one sender per slice among the
 * source replicas (Section 3.2), and moves every slice with fused HIP
 * kernels (one launch per kind of chunk the plan holds) that read it once
 * and write it to every receiver (the broadcast strategy of Section 3.1:
 * one sender, all receivers).
 *
 * On one GPU every mesh "device" is a separate buffer in the GPU's memory.
 *
 * Conventions shared by all calls
 * -------------------------------
 *  - Meshes are n-dimensional (1..8 axes).  Devices are numbered row-major
 *    over mesh coordinates: the (2,2) mesh is [[0,1],[2,3]] (Section 2.2,
 *    "Device mesh").  Pointer arrays are indexed by that number.
 *  - A spec has one letter per tensor dimension (Section 2.2, "Sharding
 *    spec"): "R" (replicated) or "S" followed by the mesh axes the dimension
 *    is split over, major to minor, e.g. "S^0RR", "RS^{01}R", "S_{0}RR",
 *    "S0 R S1".  Spaces and commas between letters are ignored.  A mesh axis
 *    may appear at most once; axes no dimension uses replicate.
 *  - For axes (a1,...,ap) a device at coordinates c holds shard number
 *    j = c[a1]*m[a2]*...*m[ap] + ... + c[ap] of the m[a1]*...*m[ap] shards.
 *  - A dimension of length l split into k shards gives shard j the range
 *    [j*floor(l/k) + min(j, l mod k), +floor(l/k) + (j < l mod k)): the first
 *    l mod k shards are one longer (66 into 4 is 17,17,16,16).  No padding.
 *  - Each device buffer is the dense C-order (row-major) array of its shard;
 *    its shape is given by reshard_plan_local_shape.  Shards of zero size are
 *    allowed and their pointer may be NULL.
 *  - Elements are opaque: only the byte size of the dtype matters, and bits
 *    are copied exactly (NaN payloads, -0 and infinities included).
 *  - Every call returns a status and never throws or aborts.  On failure
 *    reshard_last_error() describes the reason.
 */
#ifndef RESHARD_H
#define RESHARD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct reshard_plan_s reshard_plan_t;  /* opaque; created by reshard_plan */

typedef enum {
    RESHARD_OK = 0,
    RESHARD_EINVAL = 1,       /* bad argument: spec, mesh, shape, pointer, alignment */
    RESHARD_EUNSUPPORTED = 2, /* valid but beyond a compiled limit (see below) */
    RESHARD_ENOMEM = 3,       /* host or device allocation failed */
    RESHARD_EHIP = 4          /* a HIP runtime call or kernel launch failed */
} reshard_status_t;

/* Element types.  Only the byte size (1, 2, 4 or 8) is used. */
typedef enum {
    RESHARD_U8 = 0, RESHARD_I8 = 1, RESHARD_F16 = 2, RESHARD_BF16 = 3,
    RESHARD_F32 = 4, RESHARD_I32 = 5, RESHARD_F64 = 6, RESHARD_I64 = 7,
    RESHARD_U16 = 8, RESHARD_I16 = 9, RESHARD_U32 = 10, RESHARD_U64 = 11
} reshard_dtype_t;

/* reshard_plan flags */
#define RESHARD_SENDER_NAIVE 0x1u  /* lowest-indexed owner sends (Section 3.2, "Naive
                                      algorithm"); default is longest-first greedy
                                      balancing of sent bytes per device (Eq. 4). */
#define RESHARD_XCD_REMAP 0x2u     /* give each of the 8 XCDs a contiguous run of the chunk
                                      table (default: chunks start in table order, the
                                      unaligned row gather's in runs of 16 per XCD). */
#define RESHARD_TASK_ORDER 0x4u    /* keep the chunk table task by task (default: ordered by
                                      destination address -- receiver set, then offset -- so
                                      workgroups running together fill whole destination rows). */
#define RESHARD_NO_REALIGN 0x8u    /* rows whose source and destination 16-byte phases differ
                                      are copied with narrow vectors instead of being
                                      realigned into 16-byte destination slots. */
#define RESHARD_LDS_STAGING 0x10u  /* such rows are realigned by staging source words in LDS
                                      (default: two overlapping aligned loads per slot,
                                      funnel-shifted in registers). */

#define RESHARD_NO_GATHER 0x100u   /* copy every unit task separately (default: tasks that share
                                      a receiver set and cut its rows into column segments --
                                      equal and 16-byte aligned, or of any width of at least 16
                                      bytes over destination rows contiguous in runs of at least
                                      one chunk -- are written together, one
                                      workgroup gathering destination rows or 16-byte slots
                                      from all their senders). */

/* Comparison strategies (Section 3.1), for measuring what broadcast saves; at
 * most one.  Both read every slice once per receiver (R x the bytes of D) and
 * copy rows directly (no row gather, no realignment path).  Default:
 * broadcast, one read and one write per receiver. */
#define RESHARD_STRATEGY_SENDRECV 0x20u   /* the sender's slice is re-read for each receiver */
#define RESHARD_STRATEGY_ALLGATHER 0x40u  /* send/recv + all-gather: chunks go round-robin to the
                                             receivers, then (second launch) each receiver pulls
                                             the chunks it lacks from the receiver holding them */

/* Compiled limits (RESHARD_EUNSUPPORTED beyond them). */
#define RESHARD_MAX_NDIM 8
#define RESHARD_MAX_MESH_NDIM 8
#define RESHARD_MAX_BUFFERS 496    /* source + destination devices of one plan */

/* Optional tuning of the lowering; zero fields take the defaults. */
typedef struct {
    int64_t chunk_bytes;    /* source bytes per workgroup chunk (default: 4..16 KiB, sized
                               so a large plan has >= 4096 chunks, larger past 64 GiB of
                               unique data); whole vectors */
    int32_t block_threads;  /* threads per workgroup: 64, 128, 256, 512 or 1024; 0 = default:
                               256, and 512 for direct chunks whose fan-out is 2 */
    int32_t max_wgs_per_cu; /* cap on resident workgroups per CU, 2..32, enforced by reserving
                               LDS per workgroup and rounded down to an even count (a CU's
                               LDS is reserved in two halves); 0 = default, chosen per kernel
                               from its fan-out (direct chunks: 16 waves per CU at fan-out
                               <= 2, 8 above; both row-gather kinds: 64 / fan-out waves, at
                               least 8, except unaligned row gathers with one sender per row,
                               which take 32, 16 and 8 waves at fan-out 1, 2 and above, and
                               32 at any fan-out when their chunks are under 3/4 full on
                               average (rows in short runs); 32 for unaligned row gathers
                               with segments under 16 bytes at fan-out up to 4; never below
                               2 workgroups); -1 = no cap */
    int32_t gather_band;    /* row-gather chunks: column segments per band (>= 0); the chunks
                               of a row group cover one band of the destination rows after
                               another; 0 = whole rows (default) */
    int32_t reserved[3];    /* must be zero */
} reshard_tuning_t;

/*
 * Build a plan for resharding a tensor of shape[ndim] (ndim 1..8, each
 * shape[i] >= 0) with elements of `dtype` from src_mesh (src_mesh_ndim axes,
 * each >= 1) under src_spec to dst_mesh under dst_spec.
 *
 * Host only, thread-safe, no HIP call.  Computes per-device shard boxes, the
 * unit tasks (non-empty intersections of source and destination shards, each
 * with its owners and its receivers; Section 2.2 and the appendix), the
 * sender of each (flags), and the descriptor table the kernels run from.
 * The source and destination meshes are disjoint sets of buffers (Section 2.2).
 *
 * On success *out owns a new plan (free with reshard_plan_destroy).
 * Errors: EINVAL for a malformed spec, spec length != ndim, an axis outside the
 * mesh or used twice, ndim or mesh_ndim outside 1..8, a negative dimension, a
 * mesh axis < 1, NULL shape/mesh/spec/out; EUNSUPPORTED when the two meshes
 * together have more than RESHARD_MAX_BUFFERS devices, or the plan would need
 * more than 2^24 unit tasks or 2^24 workgroup chunks (automatic chunk sizes
 * grow with the tensor to stay well below; an explicit tuning.chunk_bytes can
 * exceed it, and so can a permuted layout whose rows lie so far apart that a
 * chunk holds only a few of them -- lowering stops at the first chunk past
 * the limit); ENOMEM on allocation failure.  *out is set to NULL on error.
 */
reshard_status_t reshard_plan(int ndim, const int64_t *shape, reshard_dtype_t dtype,
                              int src_mesh_ndim, const int64_t *src_mesh, const char *src_spec,
                              int dst_mesh_ndim, const int64_t *dst_mesh, const char *dst_spec,
                              unsigned flags, reshard_plan_t **out);

/* As reshard_plan, with lowering knobs (NULL = defaults).  EINVAL for a bad
 * block size, a negative chunk size, a workgroup cap outside -1, 0, 2..32, a
 * negative band or non-zero reserved fields. */
reshard_status_t reshard_plan_ex(int ndim, const int64_t *shape, reshard_dtype_t dtype,
                                 int src_mesh_ndim, const int64_t *src_mesh, const char *src_spec,
                                 int dst_mesh_ndim, const int64_t *dst_mesh, const char *dst_spec,
                                 unsigned flags, const reshard_tuning_t *tuning,
                                 reshard_plan_t **out);

/*
 * As reshard_plan_ex, with permuted local layouts on either side: the buffer
 * of every source (destination) device holds its shard with its dimensions
 * in the order src_perm (dst_perm) -- buffer dimension k is tensor
 * dimension perm[k], so the buffer is numpy.transpose(shard, perm) in dense
 * C order -- and reshard_plan_local_shape reports that order.  NULL is the
 * identity (the layout of reshard_plan).  The paper's sharding specs never
 * permute dimensions (Section 2.2, "Sharding spec"); this lets a reshard
 * also change the memory order of the tensor, e.g. [batch, seq, hidden] on
 * one side and [batch, hidden, seq] on the other.  Where the two sides are
 * contiguous along different tensor dimensions, tiles are transposed
 * through LDS (reshard_plan_transpose_chunks).
 *
 * perm arrays have ndim entries and are read during the call only.
 * Errors: those of reshard_plan_ex; EINVAL when a permutation does not
 * order 0..ndim-1; EUNSUPPORTED for a comparison-strategy flag with a
 * permuted layout.
 */
reshard_status_t reshard_plan_permuted(int ndim, const int64_t *shape, reshard_dtype_t dtype,
                                       int src_mesh_ndim, const int64_t *src_mesh, const char *src_spec,
                                       const int32_t *src_perm, int dst_mesh_ndim, const int64_t *dst_mesh,
                                       const char *dst_spec, const int32_t *dst_perm, unsigned flags,
                                       const reshard_tuning_t *tuning, reshard_plan_t **out);

/*
 * Upload the plan's descriptor, receiver and segment tables to the current
 * HIP device (one hipMalloc + synchronous copies; nothing if already done
 * on that device).  After it, reshard_execute on that device allocates and
 * copies nothing, so it can run under HIP graph capture.  Errors: EINVAL
 * for a NULL plan, ENOMEM if the allocation fails, EHIP if a HIP call
 * fails.
 */
reshard_status_t reshard_plan_upload(const reshard_plan_t *plan);

/*
 * Run the plan: fill every destination buffer from the source buffers --
 * the data movement of one cross-mesh resharding task (Section 2.2), each
 * unit task moved as a broadcast from its chosen sender to all its
 * receivers (Section 3.1), every unique slice read once (the lower bound of
 * Section 2.2).
 *
 * src_ptrs[k] (k < number of source devices) and dst_ptrs[k] (k < number of
 * destination devices) are device pointers on the current HIP device, each to
 * the dense C-order shard of that device, owned by the caller.  A pointer may
 * be NULL only if its shard is empty.  Pointers must be aligned to
 * reshard_plan_alignment() bytes.  A destination buffer must not overlap
 * another destination buffer or any source buffer; source buffers may
 * overlap one another (they are only read).  `stream` is a hipStream_t
 * (NULL = the null stream), passed as void * so this header needs no HIP
 * header and a plain C compiler can include it; hipStream_t is itself a
 * pointer to an opaque struct, so the two are the same at the ABI.
 *
 * Asynchronous and stream-ordered: it enqueues one kernel per kind of chunk
 * the plan holds (one for every workload of the paper's shapes) and returns.
 * The first call on a device uploads the descriptor table to memory the plan
 * owns (one hipMalloc + synchronous copies) unless reshard_plan_upload did;
 * later calls only launch, so they can be captured into a HIP graph.  A plan
 * may be executed any number of times, on any stream, from any number of
 * host threads at once (the first upload on a device is serialised by the
 * plan's lock); calls on different streams that write the same destination
 * buffers race, as any two kernels would.  Destroying a plan while another
 * thread still uses it, or before its launched kernels have finished, is the
 * caller's error.
 *
 * Errors: EINVAL for NULL plan or pointer arrays, a NULL or misaligned buffer
 * for a non-empty shard; ENOMEM if the table upload cannot allocate; EHIP if a
 * HIP call or the launch fails.
 */
reshard_status_t reshard_execute(const reshard_plan_t *plan, void *const *src_ptrs,
                                 void *const *dst_ptrs, void *stream);

/*
 * As reshard_execute, for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  It allocates nothing: instead of a device table owned by the
 * plan, it copies the plan's descriptor, receiver and segment tables
 * (hipMemcpyAsync on `stream`) into a fixed scratch array that the library
 * holds on every device it runs on, RESHARD_NOALLOC_MAX_TABLE_BYTES bytes,
 * for the life of the process; the kernels are reshard_execute's.  Executing
 * the same plan again on the same stream reuses the tables already there.
 *
 * Arguments, ownership and the buffers' layout are reshard_execute's.  All
 * calls on one device share its scratch array, which keeps the last call's
 * tables: calls that overlap on one device (another stream, another thread,
 * a plan destroyed and another executed while kernels still run) race, and
 * the caller must order them.  Nothing in the array needs clearing.
 *
 * Errors: those of reshard_execute, and EUNSUPPORTED when the plan's tables
 * exceed RESHARD_NOALLOC_MAX_TABLE_BYTES (every workload of the paper's
 * shapes needs at most 3.2 MiB; larger chunks shrink the table).
 */
#define RESHARD_NOALLOC_MAX_TABLE_BYTES (4u << 20)
reshard_status_t reshard_execute_noalloc(const reshard_plan_t *plan, void *const *src_ptrs,
                                         void *const *dst_ptrs, void *stream);

/* Free a plan and its device table.  A plan is built once and reused
 * because a resharding task repeats every training iteration (Section 2.2);
 * this ends that reuse.  NULL is accepted.  The caller must make sure no
 * launched execute of this plan is still running. */
void reshard_plan_destroy(reshard_plan_t *plan);

/* Shape of device `device`'s shard on side 0 (source) or 1 (destination):
 * the extent of the data slice the device holds under its mesh and spec
 * (Section 2.2, "Sharding spec"; the split of the appendix decomposition,
 * balanced for lengths the shard count does not divide).  Writes ndim values
 * to shape_out (caller-owned).  EINVAL for a bad side/device/NULL. */
reshard_status_t reshard_plan_local_shape(const reshard_plan_t *plan, int side, int64_t device,
                                          int64_t *shape_out);

/* Plan totals (any output pointer may be NULL):
 *  bytes_read    = bytes of D, each unique slice read once (the lower bound of
 *                  Section 2.2) -- or R x that under a comparison strategy;
 *  bytes_written = sum of all destination shard sizes (replicas counted);
 *  n_unit_tasks, n_descriptors (workgroup chunks), max_fanout (largest
 *  receiver count of a unit task). */
reshard_status_t reshard_plan_stats(const reshard_plan_t *plan, int64_t *bytes_read,
                                    int64_t *bytes_written, int64_t *n_unit_tasks,
                                    int64_t *n_descriptors, int64_t *max_fanout);

/* Introspection of the lowering, the chunks each unit task's broadcast is
 * cut into (Section 3.1): plan properties and chunk counts per kind. */

/* Required byte alignment of every buffer pointer passed to reshard_execute
 * (1..16), or 0 for a NULL plan. */
int64_t reshard_plan_alignment(const reshard_plan_t *plan);

/* LDS bytes per workgroup the plan's realignment chunks stage rows through
 * (0 unless RESHARD_LDS_STAGING is set and some rows need realigning), or -1
 * for a NULL plan. */
int64_t reshard_plan_lds_bytes(const reshard_plan_t *plan);

/* Number of workgroup chunks that realign rows (source and destination in
 * different 16-byte phases), or -1 for a NULL plan. */
int64_t reshard_plan_realign_chunks(const reshard_plan_t *plan);

/* Number of workgroup chunks that write whole destination rows gathered
 * from several senders whose row segments are equal and 16-byte aligned
 * (RESHARD_NO_GATHER turns them off), or -1 for a NULL plan. */
int64_t reshard_plan_gather_chunks(const reshard_plan_t *plan);

/* Number of workgroup chunks that write destination rows (contiguous, or
 * contiguous in runs of at least 2 KiB) gathered from senders whose row
 * segments have any widths and any byte alignment (uneven splits, rows in
 * different 16-byte phases; RESHARD_NO_GATHER turns them off), or -1 for a
 * NULL plan. */
int64_t reshard_plan_unaligned_gather_chunks(const reshard_plan_t *plan);

/* Of reshard_plan_unaligned_gather_chunks, the number that move 16-byte
 * units of each segment with unaligned loads and stores (one receiver,
 * segments under 2 KiB on average; a kernel of their own), or -1 for a NULL
 * plan. */
int64_t reshard_plan_unit_gather_chunks(const reshard_plan_t *plan);

/* Number of workgroup chunks that transpose tiles through LDS (tasks whose
 * source and destination layouts are contiguous along different tensor
 * dimensions), or -1 for a NULL plan. */
int64_t reshard_plan_transpose_chunks(const reshard_plan_t *plan);

/*
 * Unit task `index` (0 <= index < n_unit_tasks), in lexicographic order of the
 * slice's lower corner.  Writes lo[ndim] and hi[ndim] (the slice is
 * [lo, hi) per dimension of D), the chosen sender, all owners (senders,
 * ascending, up to senders_cap written, total in *n_senders) and all
 * receivers (ascending, up to receivers_cap written, total in *n_receivers).
 * Output pointers may be NULL when their capacity is 0.  EINVAL for a bad
 * index or NULL plan/lo/hi.
 */
reshard_status_t reshard_plan_unit_task(const reshard_plan_t *plan, int64_t index,
                                        int64_t *lo, int64_t *hi, int64_t *chosen_sender,
                                        int64_t *senders, int64_t senders_cap, int64_t *n_senders,
                                        int64_t *receivers, int64_t receivers_cap,
                                        int64_t *n_receivers);

/*
 * Run the plan's descriptor table on HOST memory with a plain loop: the same
 * table, index arithmetic and fan-out the kernels use, so the lowering can be
 * checked on a machine without a GPU.  Never called by reshard_execute.
 * src_ptrs/dst_ptrs are host pointers with the layout described above.
 * EINVAL for NULL arguments or a NULL buffer of a non-empty shard, and (text
 * starting "internal:") when a chunk would touch bytes outside its shard --
 * a lowering error the kernels would turn into a fault.
 */
reshard_status_t reshard_debug_execute_host(const reshard_plan_t *plan, void *const *src_ptrs,
                                            void *const *dst_ptrs);

/* Scheduling algorithms of Section 3.2 for the multi-host setting. */
typedef enum {
    RESHARD_SCHED_NAIVE = 0,         /* lowest-indexed owner sends; tasks in task order */
    RESHARD_SCHED_LOAD_BALANCE = 1,  /* Eq. 4 greedy: longest first to the least-loaded host,
                                        run in that order */
    RESHARD_SCHED_DFS = 2,           /* depth-first search over (next task, sender host) with
                                        per-host lower-bound pruning, max_dfs_nodes branches */
    RESHARD_SCHED_RANDOMIZED = 3,    /* greedy search with randomization: random_rounds random
                                        orders per step, keep the set busying the most hosts */
    RESHARD_SCHED_ENSEMBLE = 4       /* the better of DFS and randomized (ties: DFS) */
} reshard_sched_algo_t;

/*
 * Choose a sender and a start time for every unit task of `plan` under the
 * paper's cluster model (Section 3.2, Eq. 1-3): a task occupies its sender
 * host and all its receiver hosts for its duration; tasks sharing a host do
 * not overlap; the makespan is minimised.  Device d of the source mesh lives
 * on host d / src_devices_per_host, of the destination mesh on host
 * d / dst_devices_per_host (the meshes are disjoint, Section 2.2).  A task's
 * duration is its slice's byte count (a broadcast takes about one transfer of
 * the slice, Section 3.1), so times are in bytes at unit bandwidth.
 *
 * Host only; does not change the plan (on one GPU every task runs
 * concurrently in one kernel launch, so order only matters between hosts).
 * Writes n_unit_tasks entries to sender_out (a source device: the task's
 * lowest-indexed owner on the chosen host) and start_out, plus the makespan,
 * a lower bound (no host finishes before the work it must do) and the DFS
 * branch count.  Any output may be NULL.  random_rounds 0 means 1; seed
 * drives SplitMix64 (Steele et al., OOPSLA 2014).  EINVAL for NULL plan,
 * devices per host < 1, negative budgets or an unknown algorithm.
 */
reshard_status_t reshard_schedule(const reshard_plan_t *plan, int64_t src_devices_per_host,
                                  int64_t dst_devices_per_host, reshard_sched_algo_t algo,
                                  int64_t max_dfs_nodes, int64_t random_rounds, uint64_t seed,
                                  int64_t *sender_out, int64_t *start_out, int64_t *makespan_out,
                                  int64_t *lower_bound_out, int64_t *dfs_nodes_out);

/*
 * Latency of one training iteration under the pipeline schedules of Section
 * 4, with cross-mesh resharding between stages: `stages` stages run
 * `microbatches` micro-batches; stage s (0-based) runs w forwards, then
 * alternately one backward and one forward, then the remaining backwards,
 * with w = stages - s (1F1B, eager = 0) or w = 2(stages - s) - 1
 * (eager-1F1B, eager = 1), capped at microbatches.  A forward needs the
 * previous stage's forward of the same micro-batch plus a transfer of
 * t_comm_fwd; a backward needs the next stage's backward plus t_comm_bwd (the
 * last stage's backward follows its own forward).  Transfers overlap with
 * computation; with serial_links != 0 transfers on one directed stage pair go
 * one at a time.  Writes the latency and, per stage, the peak number of
 * micro-batches whose forward is done and backward is not (stages entries).
 * Host only.  EINVAL for stages or microbatches < 1 or a negative time.
 */
reshard_status_t reshard_pipeline_simulate(int32_t stages, int32_t microbatches, int32_t eager,
                                           double t_fwd, double t_bwd, double t_comm_fwd,
                                           double t_comm_bwd, int32_t serial_links,
                                           double *latency_out, int32_t *peak_live_out);

/* Text of the last error on the calling thread ("" if none).  Not an
 * operation of the paper: the error report of this interface, which never
 * throws across it.  Never NULL; owned by the library; valid until the
 * next call on the same thread. */
const char *reshard_last_error(void);

/* Library version string, e.g. "0.1.0". */
const char *reshard_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RESHARD_H */
