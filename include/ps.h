/*
 * ps.h -- C ABI of an ASGD parameter server held in one gfx950 GPU's memory.
 *
 * Model (GaDei, arXiv 1611.06213):
 *   - Learners push gradients to the server and pull weights from it; they
 *     never talk to each other (Sec. 2.1, Fig. "design_base"; Sec. 4.1).
 *   - Asynchronous SGD: the server applies every gradient it receives, in the
 *     order received, each as one step theta <- theta - alpha * grad
 *     (Eq. "asgd" with the step of Eq. "gd", Sec. 2.1).
 *   - The server's weights carry a scalar timestamp that grows by one per
 *     applied gradient; the staleness of a gradient is the server timestamp
 *     when it is applied minus the timestamp of the weights its learner held
 *     (Sec. 2.1).
 *   - Gradients wait in a producer-consumer queue with a fixed number of
 *     slots; each is applied exactly once and a full queue refuses the
 *     producer (Sec. 4.1; Lemma 1 and Theorem 2, Sec. 4.2).
 *   - A learner whose copy already carries the server's timestamp skips its
 *     pull (Sec. 4.1).
 *
 * Design on one GPU:
 *   - The library owns the fp32 weights w[n] (and, with momentum, the fp32
 *     velocity v[n]) in device memory.
 *   - ps_push only records a descriptor; it copies nothing. The gradient
 *     stays in the caller's device buffer until the apply that consumes it.
 *   - ps_apply_pending folds all pending gradients into w in one pass over
 *     memory: for each coordinate, the K gradients are applied one after the
 *     other, oldest first, with the same roundings as K separate steps.
 *   - All device work is enqueued, asynchronously, on one HIP stream in call
 *     order (the stream set by ps_set_stream; the null stream by default).
 *     A pull therefore sees every gradient applied by earlier calls and no
 *     gradient still pending.
 *
 * Arithmetic per coordinate and per applied gradient g (binary32, each
 * operation rounded to nearest even, no fused multiply-add):
 *   momentum == 0:  p = lr*g;  w = w - p
 *   momentum != 0:  t = m*v;  v = t + g;  p = lr*v;  w = w - p   (v starts +0)
 * A bf16 gradient is widened exactly to fp32 first. A bf16 pull writes w
 * rounded to nearest even bf16.
 *
 * Threading: every call takes the handle's lock, so several host threads
 * may use one server, e.g. a push thread per learner beside a server thread
 * that applies and serves pulls (the paper's thread layout, Sec. 4.1).
 * Calls are served one at a time in lock order, and device work is enqueued
 * in that order. ps_sync waits without holding the lock. ps_destroy must
 * not race other calls on the handle. Distinct handles are independent.
 *
 * Pointers named "device" must point to device memory (hipMalloc or torch
 * CUDA tensors) on the device that was current at ps_create. Any alignment is
 * accepted and gives identical results: 16-byte-aligned buffers take the
 * widest vector path, 8-byte-aligned bf16 buffers a narrower one, others a
 * scalar path. Buffers that start on 256-byte (better: 2 MiB) boundaries
 * stream fastest.
 *
 * Status codes: every int-returning call returns PS_OK (0) or a negative
 * PS_E* code; ps_last_error() then describes the failure (per thread).
 * Argument errors (PS_EINVAL, PS_EFULL, PS_ESTATE) are found before any
 * state changes or device work. A PS_EHIP from a launch means the device or
 * runtime has failed: the gradients of an apply whose kernels were all
 * enqueued count as applied, but if an apply over gradients of both dtypes
 * fails between its two launches the weights hold part of the batch, and
 * the handle should only be destroyed.
 */
#ifndef GADEI_PS_H
#define GADEI_PS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ps_server ps_server;

enum {
    PS_OK = 0,
    PS_EINVAL = -1,  /* bad handle, id, pointer, dtype or size              */
    PS_EFULL = -2,   /* push on a full queue; nothing was enqueued          */
    PS_ENOMEM = -3,  /* device or host allocation failed                    */
    PS_EHIP = -4,    /* a HIP runtime call or kernel launch failed          */
    PS_ESTATE = -5,  /* call not allowed in the current state               */
    PS_EIO = -6      /* checkpoint file could not be written, read or trusted */
};

enum { PS_F32 = 0, PS_BF16 = 1 };

/* Queue modes (ps_set_queue_mode). */
enum {
    PS_QUEUE_FIFO = 0,        /* one queue of `depth` slots, push-call order   */
    PS_QUEUE_ROUND_ROBIN = 1  /* a queue per learner, served round-robin      */
};

#define PS_MAX_QUEUE_DEPTH 64   /* K: gradients folded by one apply         */
#define PS_MAX_REPLICAS 64      /* replica buffers written by one pull call */
#define PS_MAX_LEARNERS 65536   /* learner ids are 0 .. PS_MAX_LEARNERS-1   */
#define PS_STALENESS_BINS 64    /* histogram bins; the last one is ">= 63"  */
#define PS_MAX_ROWS 4096        /* buffers one ps_alloc_rows call may carve */

typedef struct ps_stats {
    uint64_t timestamp;        /* applied gradients so far (Sec. 2.1)       */
    uint64_t pushes_accepted;
    uint64_t pushes_rejected;  /* PS_EFULL returns                          */
    uint64_t pushes_applied;
    uint64_t pushes_dropped;   /* discarded by ps_drop_learner              */
    uint64_t applies;          /* apply calls that launched device work     */
    uint64_t pulls;            /* replica refreshes requested               */
    uint64_t pulls_skipped;    /* ... of which skipped as already current   */
    uint64_t staleness_max;
    uint64_t staleness_sum;
    uint64_t staleness_hist[PS_STALENESS_BINS];
} ps_stats;

/* Create a server for n_params fp32 weights with learning rate lr (alpha in
 * Eq. "gd") and heavy-ball momentum (0 disables it and allocates no v).
 * Allocates w (and v) on the current device; w starts at zero, v at +0,
 * timestamp 0, queue depth PS_MAX_QUEUE_DEPTH / 2 = 32, pull skipping on.
 * Returns NULL on failure (n_params == 0 or above 2^48, lr or momentum not
 * finite, allocation failure); see ps_last_error(). */
ps_server *ps_create(size_t n_params, float lr, float momentum);

/* Wait for the server's stream, then free w and v and the handle. NULL is a
 * no-op. Pending (unapplied) gradients are dropped. */
void ps_destroy(ps_server *ps);

/* Push the fp32 gradient grad[n_params] (device pointer) of learner
 * learner_id (Sec. 2.1, Eq. "asgd"). Records it at the tail of the FIFO; no
 * data moves. The buffer is borrowed: the caller must not write or free it
 * until the apply that consumes it has completed on the server's stream.
 * Returns PS_EFULL, with nothing enqueued, when the queue holds its depth of
 * gradients (Sec. 4.1, Theorem 2): apply, then push again. PS_EINVAL when
 * the buffer overlaps the server's w or v. */
int ps_push(ps_server *ps, int learner_id, const void *grad);

/* ps_push for a gradient of the given dtype (PS_F32 or PS_BF16; a bf16
 * gradient holds n_params 16-bit values). */
int ps_push_dtype(ps_server *ps, int learner_id, const void *grad, int dtype);

/* ps_push_dtype for a gradient that a producer may still be writing on
 * another stream (the paper's push thread works on its own stream, Sec.
 * 4.1): `ready_event` is a hipEvent_t the producer recorded after its last
 * write, and the apply that consumes the gradient makes the server's stream
 * wait for it on the device -- the host never blocks. NULL = ready now. The
 * event must stay valid until that apply has been enqueued. */
int ps_push_async(ps_server *ps, int learner_id, const void *grad, int dtype, void *ready_event);

/* Apply the pending gradients -- FIFO mode: all of them, oldest first;
 * round-robin mode: up to `depth` in service order (ps_set_queue_mode) --
 * each as one step of Eq. "asgd", and remove them from their queues.
 * Enqueues one kernel per run of equal-dtype gradients (one in the usual
 * case) on the server's stream; returns without waiting. The timestamp grows by the number applied; staleness of each is
 * recorded (ps_last_staleness, ps_last_applied, ps_get_stats). With nothing
 * pending no device work is done and the last-apply queries report 0. */
int ps_apply_pending(ps_server *ps);

/* Synchronous SGD step (Eq. "ssgd", Sec. 2.1): average the pending
 * gradients -- the caller pushes one per learner, lambda in all -- summed per
 * coordinate in push order from +0 and divided by their count (correctly
 * rounded division), and apply the average as one step of Eq. "gd" (the
 * heavy-ball form when momentum != 0). The timestamp grows by one; each
 * gradient's staleness is recorded as for ps_apply_pending. All pending
 * gradients must share one dtype (PS_EINVAL otherwise, nothing applied). An
 * empty queue is a no-op. Asynchronous on the server's stream. */
int ps_apply_sync(ps_server *ps);

/* Pull: write the current weights into the learner's replica buffer
 * dst[n_params] (device, fp32). Asynchronous on the server's stream; the copy
 * sees every apply issued before it. Skipped (no device work) when the same
 * learner last pulled into the same buffer with the same dtype at the current
 * timestamp (Sec. 4.1). dst must not overlap a pending gradient; overlapping
 * w or v is refused with PS_EINVAL. */
int ps_pull(ps_server *ps, int learner_id, void *dst);

/* Pull for n learners at once: learner_ids[i] into dsts[i], all in dst_dtype
 * (PS_F32, or PS_BF16 = round to nearest even). One fan-out kernel writes
 * every replica that is not skipped, reading w from HBM once (it walks w in
 * tiles that stay cached while the replicas of a tile are written).
 * 0 <= n <= PS_MAX_REPLICAS; the buffers that are written must be distinct,
 * and none may overlap w or v (PS_EINVAL, nothing written). */
int ps_pull_many(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype);

/* ps_apply_pending followed by ps_pull_many, in one call; the result is
 * identical to the two calls in sequence. Up to the fusion limit (see
 * ps_set_pull_fusion) the replicas are written from the same pass that
 * updates w, so w is not read again; above it the apply kernel is followed
 * by the tiled fan-out, which serves many replicas faster than one pass.
 * With lock-free pulls on (ps_set_pull_stream) and replicas to write, the
 * call first makes the server's stream wait for the lock-free pulls already
 * enqueued, so none of them can overwrite a replica this call marks
 * current. */
int ps_apply_pull(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype);

/* Largest replica count ps_apply_pull writes from the apply pass itself
 * (0..PS_MAX_REPLICAS), or -1 (default) to choose per call: one replica
 * always, up to 4 when the apply folds at most 16 gradients, up to 6 when it
 * folds at most 8 into a vector of fewer than 20M coordinates (measured
 * faster there; with more gradients or replicas the separate fan-out is).
 * Results are identical either way. PS_EINVAL for other values. */
int ps_set_pull_fusion(ps_server *ps, int max_replicas);

/* Use hip_stream (a hipStream_t; NULL = the null stream) for all later device
 * work. The caller orders it against work already on the previous stream. */
int ps_set_stream(ps_server *ps, void *hip_stream);

/* Record `event` (a hipEvent_t) on the server's stream after all work
 * enqueued so far: when it completes, every gradient consumed by an earlier
 * apply may be overwritten and every earlier ordered pull is complete. A
 * producer stream can wait for it instead of the host (double buffering). */
int ps_record(ps_server *ps, void *event);

/* Lock-free pulls (the paper's default HogWild! mode, Sec. 4.1): with a
 * non-NULL hip_stream, ps_pull / ps_pull_many run there, not ordered after
 * applies on the server's stream, so a pull concurrent with an apply may
 * write, coordinate by coordinate, the weights from before or after it
 * (each coordinate is one of the two; the replica as a whole may mix them).
 * The caller orders such pulls against earlier applies itself if it needs
 * to (ps_record + hipStreamWaitEvent). A lock-free pull never makes a copy
 * count as current, so the next pull of that learner is not skipped; the
 * learner's timestamp is taken at the call. ps_apply_pull still orders its
 * pull after its apply. NULL (default) restores ordered pulls -- the
 * paper's read-write-lock option. Waits for
 * earlier lock-free pulls before switching; ps_sync, ps_set_weights,
 * ps_save, ps_load and ps_destroy wait for them too. */
int ps_set_pull_stream(ps_server *ps, void *hip_stream);

/* Queue depth K, 1..PS_MAX_QUEUE_DEPTH: the FIFO's slots, and the most
 * gradients one asynchronous apply takes. PS_ESTATE if (FIFO mode) more
 * gradients are pending than the new depth. */
int ps_set_queue_depth(ps_server *ps, int depth);

/* Queue topology. PS_QUEUE_FIFO (default): one queue of `depth` slots in
 * push-call order. PS_QUEUE_ROUND_ROBIN: each learner has its own queue of
 * slots_per_learner slots (1..PS_MAX_QUEUE_DEPTH) -- the paper's lambda
 * single-producer single-consumer queues with a fixed number of slots per
 * learner (Sec. 4.1) -- and a push on a full one returns PS_EFULL (Lemma 1).
 * The server visits learners in increasing id order, cyclically, starting
 * after the learner it served last, and takes one gradient per visit of a
 * non-empty queue (Sec. 4.1); an asynchronous apply takes up to `depth`
 * gradients this way and leaves the rest queued. A synchronous step takes
 * the oldest gradient of every waiting learner, in increasing id, and
 * returns PS_ESTATE if more than PS_MAX_QUEUE_DEPTH learners wait. PS_ESTATE
 * if any gradient is pending; slots_per_learner is ignored for FIFO. */
int ps_set_queue_mode(ps_server *ps, int mode, int slots_per_learner);

/* How the apply kernels sweep the weights: 2^fronts_log2 evenly spaced
 * fronts (0..3), or -1 (default) to choose per apply from the buffers'
 * offsets within 2 MiB -- four fronts when at least 8 buffers take part and
 * more than half of the gradient, w and v buffers share one 4 KiB offset (as
 * separately allocated, 2 MiB-aligned buffers do), one front otherwise
 * (ps_alloc_rows buffers). Results are identical either way; only the
 * order in which the grid visits coordinates changes. */
int ps_set_fronts(ps_server *ps, int fronts_log2);

/* Override the launch shape of the apply (Eq. "asgd") and synchronous-step
 * (Eq. "ssgd") kernels, which is otherwise chosen per call from the number of
 * gradients, momentum, the gradient type and, for shallow applies, the
 * vector's length (tables measured at the VGG-16, Mixed and Text-CNN sizes):
 * blocks_per_cu 1..4 caps the resident 256-thread blocks per compute unit, 0
 * lifts the cap, -1 restores the library's choice; group 4, 8, 12, 16, 24 or
 * 32 sets how many gradients' loads are issued together (the synchronous step
 * takes 16 for 24 and 32), 0 restores the library's choice. Results are
 * identical for every shape; only speed changes. For callers tuning other
 * sizes. PS_EINVAL for other values, setting unchanged. */
int ps_set_launch_shape(ps_server *ps, int blocks_per_cu, int group);

/* Enable (1) or disable (0) skipping of pulls that are already current. */
int ps_set_pull_skip(ps_server *ps, int enabled);

/* Reset the server to start from src[n_params] (device, fp32): w := src,
 * v := +0, timestamp := 0, every learner holds timestamp 0, pull history and
 * statistics cleared. PS_ESTATE if gradients are pending; PS_EINVAL if src
 * overlaps w or v. Asynchronous. */
int ps_set_weights(ps_server *ps, const float *src);

/* Device pointers to w[n_params] and v[n_params] (NULL without momentum).
 * Owned by the server; valid until ps_destroy. Reading them is ordered by the
 * server's stream. */
const float *ps_weights(const ps_server *ps);
const float *ps_velocity(const ps_server *ps);

size_t ps_num_params(const ps_server *ps);
uint64_t ps_timestamp(const ps_server *ps);
int ps_pending(const ps_server *ps);

/* Staleness of each gradient applied by the most recent apply call
 * (ps_apply_pending, ps_apply_pull, ps_apply_sync), in the order applied.
 * Writes min(count, cap) values to out and returns count (or a negative
 * status). */
int ps_last_staleness(const ps_server *ps, int64_t *out, int cap);

/* Learner ids of the gradients applied by the most recent apply call, in
 * the order applied. Writes min(count, cap) ids and returns count (or a
 * negative status). */
int ps_last_applied(const ps_server *ps, int *learner_ids, int cap);

/* A learner died (Sec. 4.3): discard its queued gradients -- its borrowed
 * buffers may be gone with it -- and keep every other gradient in order. The
 * server holds no other per-learner state that the others depend on, so
 * training continues with the live learners. Returns the number dropped
 * (>= 0) or a negative status. */
int ps_drop_learner(ps_server *ps, int learner_id);

/* A learner died (Sec. 4.3) while its gradients sat in the server's own
 * slots (ps_alloc_rows rows, which outlive the learner): the server is
 * stateless, so those gradients stay queued and are applied exactly once,
 * in their turn (Theorem 2, Sec. 4.2), like everyone else's. Later pushes
 * and pulls under learner_id are refused with PS_ESTATE, until
 * ps_set_weights or ps_load starts a new run. Returns how many of its
 * gradients are still queued (>= 0), or a negative status: PS_ESTATE, with
 * nothing changed, when one of them lies outside the server's rows (a
 * borrowed buffer may be gone with the learner: use ps_drop_learner). */
int ps_retire_learner(ps_server *ps, int learner_id);

/* Checkpoint (Sec. 4.3: the server checkpoints its parameters so that a
 * restart resumes from the last checkpoint). ps_save writes w, v, the
 * timestamp, the queue configuration (mode, depth, slots per learner), the
 * round-robin position and every learner's timestamp to `path` (waits for
 * the server's stream and lock-free pulls first); ps_load restores them
 * into a server created with the same n_params, lr and momentum and set to
 * the same queue configuration, after checking the whole file (format
 * version, sizes, a checksum over header and data) -- on any failure the
 * server is unchanged. Pull history and statistics start afresh after a
 * load (learners pull again after a restart). Both need an empty queue
 * (PS_ESTATE otherwise); file errors give PS_EIO, mismatched servers
 * (sizes, lr, momentum or queue configuration) PS_EINVAL. Continuing from a
 * loaded checkpoint gives the bits of the uninterrupted run. */
int ps_save(ps_server *ps, const char *path);
int ps_load(ps_server *ps, const char *path);

/* Server-owned device buffers for gradients or replicas: the paper's queue
 * slots, which the server holds and learners fill (Sec. 4.1). Allocates
 * `count` (1..PS_MAX_ROWS) buffers of n_params values of `dtype` in one
 * device allocation and writes their addresses to rows[0..count). Rows of
 * 2 MiB or more are 1.75 MiB apart beyond their 2 MiB-rounded size: row i
 * starts at ((i + 2) * 1.75 MiB) mod 2 MiB past a 2 MiB boundary, and v
 * sits 1.75 MiB past w's 2 MiB-rounded end (w on a 2 MiB boundary).
 * Smaller rows are packed on 4 KiB boundaries. An apply then streams its
 * gradients, w and v from spread-out addresses, which the DRAM serves
 * fastest of the layouts measured. Buffers allocated one by one
 * (2 MiB-aligned, all at one phase) are served slower; for them the apply
 * kernels switch to a schedule that recovers part of the difference.
 * Contents are uninitialised. The buffers belong to the server
 * until ps_free_rows(ps, rows[0]) or ps_destroy. PS_ENOMEM if the device
 * allocation fails. */
int ps_alloc_rows(ps_server *ps, int count, int dtype, void **rows);

/* Free the buffers of one ps_alloc_rows call, named by its first row, after
 * waiting for the server's streams. PS_ESTATE (nothing freed) if a pending
 * gradient lies in them; PS_EINVAL if first_row is not such a row. */
int ps_free_rows(ps_server *ps, void *first_row);

/* Learners in their own processes (Sec. 4.1, 4.3: each learner and the
 * server has its own address space and all of them map one shared region
 * holding the gradient slots and the weights). On one GPU the shared region
 * is the server's rows, shared through HIP IPC.
 *
 * ps_export_rows: a handle (PS_IPC_HANDLE_BYTES opaque bytes written to
 * `handle`) for the device allocation holding the rows of one
 * ps_alloc_rows call, named by its first row, and the offset of that row in
 * the allocation. Another process on the same device passes both to
 * ps_import_rows. The rows stay the server's: they are freed by
 * ps_free_rows or ps_destroy, after which importers must not touch them.
 * PS_EINVAL if first_row is not the first row of a row set. */
#define PS_IPC_HANDLE_BYTES 64
int ps_export_rows(ps_server *ps, void *first_row, void *handle, size_t *offset);

/* Learner side, in another process, with the server's device current: map
 * the exported allocation and write the address of its first row (rows
 * follow at the stride the server's ps_alloc_rows reported). The learner
 * writes gradients into its slots and reads replicas there; every write must
 * have completed on the device before the server is told to push it.
 * PS_EINVAL if offset lies outside the allocation or the row set is already
 * imported in this process (import once, release once); PS_EHIP if the
 * handle cannot be opened. ps_release_rows waits for this process's device
 * work, then unmaps; PS_EINVAL for a row not imported here. */
int ps_import_rows(const void *handle, size_t offset, void **first_row);
int ps_release_rows(void *first_row);

/* One call of the hot path, for ps_run. */
enum {
    PS_OP_PUSH = 0,        /* ps_push_dtype(learner_id, grad, dtype)                 */
    PS_OP_APPLY = 1,       /* ps_apply_pending                                        */
    PS_OP_APPLY_SYNC = 2,  /* ps_apply_sync                                           */
    PS_OP_PULL = 3,        /* ps_pull_many(count, learner_ids, dsts, dtype)           */
    PS_OP_APPLY_PULL = 4   /* ps_apply_pull(count, learner_ids, dsts, dtype)          */
};
typedef struct ps_op {
    int kind;                  /* PS_OP_*                                              */
    int learner_id;            /* PS_OP_PUSH                                           */
    int dtype;                 /* gradient dtype (push) or replica dtype (pulls)       */
    int count;                 /* replicas (pulls)                                     */
    const void *grad;          /* device gradient (push)                               */
    const int *learner_ids;    /* count ids (pulls)                                    */
    void *const *dsts;         /* count device replica buffers (pulls)                 */
} ps_op;

/* Run a script of hot-path calls in order, each exactly as the call it
 * names (same validation, results and errors), under one acquisition of
 * the handle's lock -- the server loop of Sec. 4.1 driven from a prepared
 * schedule without a host-language round trip per call. Stops at the first
 * call that does not return PS_OK (a full queue included) and returns its
 * status; *done (may be NULL) receives the number of calls completed.
 * PS_EINVAL for an unknown kind or ops == NULL with count > 0. */
int ps_run(ps_server *ps, const ps_op *ops, int count, int *done);

/* A script captured once as a HIP graph and replayed, for launch-bound
 * loops (small vectors, one gradient per apply): a replay enqueues all of
 * the script's kernels at once, without a launch per kernel.
 *
 * ps_graph_create: the script's calls are made as by ps_run, but their
 * kernels are captured into a graph on the server's stream instead of
 * running, and the server's host state is left as it was: nothing has run.
 * The script is copied; its gradient and replica buffers must stay valid
 * while the graph lives.
 *
 * ps_graph_launch: the calls again, planned and committed on the host as
 * by ps_run (timestamps, staleness, pull history, statistics), and the graph
 * enqueued on the server's stream, ordered with every other call. The
 * result is identical to ps_run of the same script. Every launch checks that
 * the calls would now launch exactly the captured kernels (same buffers,
 * gradients per apply, replicas written, launch shapes); if not -- say a
 * pull that was written at capture would now be skipped -- it returns
 * PS_ESTATE and changes nothing. A call of the script that fails returns
 * its status and changes nothing either.
 *
 * Both need a server stream other than the legacy null stream
 * (ps_set_stream), ordered pulls (no ps_set_pull_stream) and an empty queue
 * (PS_ESTATE otherwise); scripts start from an empty queue. While
 * ps_graph_create runs, no other thread may enqueue work on that stream
 * (it is being captured). PS_EINVAL for a
 * bad script, a script that launches nothing, or a graph of another
 * server. Destroy graphs before their server; a graph is launched only on
 * the server it was created for. ps_graph_destroy waits for the graph's
 * last launch to finish. */
typedef struct ps_graph ps_graph;
int ps_graph_create(ps_server *ps, const ps_op *ops, int count, ps_graph **graph);
int ps_graph_launch(ps_server *ps, ps_graph *graph);
void ps_graph_destroy(ps_graph *graph);

/* Block until all work enqueued by the server has completed. */
int ps_sync(ps_server *ps);

int ps_get_stats(const ps_server *ps, ps_stats *out);

/* Message for the last failed call on this thread ("" if none). */
const char *ps_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GADEI_PS_H */
