/*
 * dd.h -- batched what-if simulation of trace-derived task dependency graphs
 * on AMD Instinct MI355X (gfx950).
 *
 * The library answers "what if" questions the way Daydream does (Zhu,
 * Phanishayee, Pekhimenko, arXiv 2006.03318): a kernel-granularity task
 * graph recorded from one training iteration is transformed (tasks scaled,
 * removed, dependencies switched) and then simulated to predict the new
 * iteration time.  Here thousands of transformed variants of one graph are
 * simulated in one batch on the GPU.
 *
 * Semantics (the simulation of Sec. 4.1, Algorithm 1, "Daydream's Simulation
 * Algorithm"; task fields of Sec. 4.2.1; dependency types of Sec. 4.2.2):
 *   every task u has an execution thread (a CPU thread, a GPU stream or a
 *   communication channel), a duration d_u and a gap g_u (CPU time between
 *   the end of u and the next task on its thread), all int64 nanoseconds.
 *   Parents of u are its dependency in-edges plus the previous task on its
 *   thread.  With release R_p = start_p + d_p + g_p,
 *       start_u  = max(0, max over parents p of R_p)
 *       finish_u = start_u + d_u
 *       makespan = max over tasks not removed of finish_u   (0 if none)
 *   which is what Algorithm 1 computes: every child's start is raised to the
 *   parent's start + duration + gap, and tasks on one thread run in their
 *   recorded order (that order does not change between executions,
 *   Sec. 4.2.2).
 *
 * Transformations per variant (Sec. 4.4, graph-transformation primitives):
 *   shrink/scale: task of class c in variant v gets duration
 *                 floor(d * p / q) with (p, q) = scale[c][v];
 *   Remove:       a removed task gets duration 0 and gap 0, which is the
 *                 same as unlinking it and connecting each predecessor to
 *                 each successor; its start = finish = the time all its
 *                 inputs are available; it is left out of the makespan;
 *   re-route:     each dependency edge has a class k < 64; edges of class k
 *                 exist in variant v only if bit k of edge_on[v] is set
 *                 (tasks moved to another thread or re-ordered on a
 *                 channel are expressed by such edges).
 *   Gaps are never scaled.
 *
 * Conventions for every call:
 *   - All functions return dd_status; DD_OK (0) on success.  On failure
 *     dd_last_error() gives a message (per host thread) and no output
 *     handle is created.
 *   - Input arrays may be host or device pointers (each one independently);
 *     they are copied during the call and remain owned by the caller.
 *   - Output arrays of dd_simulate_batch are device pointers owned by the
 *     caller; the library never frees them.
 *   - Handles are owned by the library until the matching *_free.  A handle
 *     keeps device memory, released on the stream it was created on, which
 *     must stay valid until the handle is freed.  A handle may be used on
 *     any stream: the library records an event after each use on a stream
 *     other than the handle's own, and *_free makes the handle's stream wait
 *     for those events before its memory can be handed out again.  Released
 *     device memory stays in a cache of the library, kept per device and
 *     stream, and is handed out again to later calls on that same stream
 *     (stream order makes the reuse safe); it returns to the device when an
 *     allocation would otherwise fail, on dd_release_cache(), or at process
 *     exit.
 *   - `stream` is a hipStream_t (NULL = default stream).  Work is
 *     stream-ordered.  Input validation is synchronous: load, levelize and
 *     apply_transforms wait for their own device checks before returning.
 *     dd_simulate_batch is asynchronous; a device fault surfaces as DD_EHIP
 *     from the same or a later call.
 *   - Limits: 0 <= n < 2^31, n_threads >= 1, edges < 2^31, edge classes < 64,
 *     task classes < 65536, durations and gaps in [0, 2^62).
 */
#ifndef DD_H
#define DD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DD_OK = 0,
    DD_EINVAL = 1,     /* bad argument: NULL, out-of-range index or size, negative time */
    DD_ECYCLE = 2,     /* dependencies plus thread order contain a cycle */
    DD_ECHAIN = 3,     /* thread order is not one simple chain per thread */
    DD_ERANGE = 4,     /* scaled times could overflow int64 */
    DD_ENOMEM = 5,     /* device allocation failed */
    DD_EHIP = 6,       /* HIP runtime error */
    DD_EMISMATCH = 7,  /* handles from different graphs, or a variant uses an
                          edge class the schedule was not built for */
    DD_ELIMIT = 8      /* a fixed capacity of a device path was exceeded */
} dd_status;

typedef struct dd_graph dd_graph;
typedef struct dd_sched dd_sched;
typedef struct dd_variants dd_variants;

/* A duration scale p/q: p >= 0, q >= 1. */
typedef struct { int32_t p, q; } dd_ratio;

#define DD_LEVELS 0   /* steps = Kahn topological levels (longest hop path) */
#define DD_PHASES 1   /* steps = phases (longest path counting only edges
                         between different threads); one step holds one
                         contiguous run of each thread's tasks */

/*
 * dd_graph_load -- the task graph G(V, E) of Sec. 4.2 (tasks, Sec. 4.2.1;
 * dependencies, Sec. 4.2.2).
 *   n            number of tasks.
 *   n_threads    number of execution threads; thread ids are 0..n_threads-1.
 *   in_ptr       int64 [n+1], CSR offsets of dependency in-edges per task;
 *                in_ptr[0] == 0, non-decreasing.
 *   in_src       int32 [in_ptr[n]], source task of each in-edge.
 *   edge_cls     uint8 [in_ptr[n]], class (< 64) of each edge; NULL = 0.
 *   thread_prev  int32 [n], previous task on the same thread, -1 for the
 *                first; each thread must form one chain.
 *   thread_id    int32 [n], execution thread of each task.
 *   dur_ns       int64 [n], durations.   gap_ns  int64 [n], gaps.
 *   node_cls     uint16 [n], transform class of each task; NULL = 0.
 * Validates everything (DD_EINVAL, DD_ECHAIN, DD_ECYCLE for a self loop or
 * a dependency that goes backwards along one thread, DD_ERANGE), ranks the
 * thread chains, drops dependencies between tasks of the same thread (the
 * thread order already implies them) and builds the cross-thread edge lists
 * in both directions.  *out receives the handle.
 */
dd_status dd_graph_load(int32_t n, int32_t n_threads,
                        const int64_t *in_ptr, const int32_t *in_src, const uint8_t *edge_cls,
                        const int32_t *thread_prev, const int32_t *thread_id,
                        const int64_t *dur_ns, const int64_t *gap_ns, const uint16_t *node_cls,
                        void *stream, dd_graph **out);

/*
 * dd_graph_load_ex -- dd_graph_load with flags.
 *   DD_LOAD_SHARED_THREADS  a thread may hold several chains: tasks with
 *       thread_prev == -1 other than the first, and chains that share a
 *       thread, have no recorded order among themselves (for example the
 *       push and pull slices a what-if recipe inserts on a communication
 *       channel, Sec. 5.1 P3).  Their order is decided while simulating, by
 *       the schedule() rule of Sec. 4.4 ("Schedule"), so such a graph is
 *       simulated only by dd_simulate_policy; dd_levelize and
 *       dd_runtime_breakdown return DD_EINVAL for it.  Each task still has at
 *       most one thread successor (DD_ECHAIN otherwise), and dependencies
 *       between tasks of one thread are kept (no thread order implies them).
 * flags == 0 is dd_graph_load.  Unknown flag bits: DD_EINVAL.
 */
#define DD_LOAD_SHARED_THREADS 1u
dd_status dd_graph_load_ex(int32_t n, int32_t n_threads,
                           const int64_t *in_ptr, const int32_t *in_src, const uint8_t *edge_cls,
                           const int32_t *thread_prev, const int32_t *thread_id,
                           const int64_t *dur_ns, const int64_t *gap_ns, const uint16_t *node_cls,
                           uint32_t flags, void *stream, dd_graph **out);

/*
 * dd_levelize -- topological schedule of the graph restricted to the edge
 * classes in `active_edge_classes` (bit k = class k; thread order is always
 * present), computed on the GPU with Kahn's algorithm (the reference counts
 * and frontier of Algorithm 1, processed a whole frontier at a time).
 *   mode == DD_LEVELS: step of a task = its Kahn level.
 *   mode == DD_PHASES: step = its phase; every step consists of one
 *                      contiguous run of tasks per thread at most, and all
 *                      cross-thread inputs of a step come from earlier steps.
 * *n_steps_out (may be NULL) receives the number of steps.  DD_ECYCLE if
 * the active dependencies plus thread order contain a cycle.
 */
dd_status dd_levelize(const dd_graph *g, uint64_t active_edge_classes, int32_t mode,
                      void *stream, dd_sched **out, int64_t *n_steps_out);

/*
 * dd_apply_transforms -- per-variant transform tables (Sec. 4.4 primitives).
 *   n_variants   V >= 1.
 *   n_cls        rows of `scale`; must exceed every node_cls of the graph.
 *   scale        dd_ratio [n_cls][V]; NULL = all 1/1.
 *   remove_bits  uint32 [n][ceil(V/32)]; bit v%32 of word v/32 of row u set =
 *                task u removed in variant v; NULL = none removed.
 *   edge_on      uint64 [V]; bit k = edges of class k present; NULL = all.
 * DD_EINVAL for p < 0 or q < 1, DD_ERANGE if a scaled time could overflow.
 */
dd_status dd_apply_transforms(const dd_graph *g, int32_t n_variants, int32_t n_cls,
                              const dd_ratio *scale, const uint32_t *remove_bits,
                              const uint64_t *edge_on, void *stream, dd_variants **out);

/*
 * dd_simulate_batch -- simulate every variant (the hot path).
 *   d_finish    device int64 [n][V] (task-major, variant-minor), required
 *               unless n == 0: finish time of each task in each variant.
 *   d_start     device int64 [n][V] or NULL: start times.
 *   d_makespan  device int64 [V], required: iteration time of each variant.
 * All three handles must come from the same graph; every edge class some
 * variant switches on must be in the schedule's active classes
 * (DD_EMISMATCH otherwise).
 */
dd_status dd_simulate_batch(const dd_graph *g, const dd_sched *sched, const dd_variants *var,
                            int64_t *d_finish, int64_t *d_start, int64_t *d_makespan,
                            void *stream);

/*
 * dd_simulate_batch_vs -- dd_simulate_batch with an explicit launch shape.
 *   variants_per_wg  variants that each workgroup owns for the whole
 *                    schedule: 0 = chosen by the library (as
 *                    dd_simulate_batch), or 1, 2, 4, 8, 16;
 *                    -1, -2, -4, -8 = the few-variant path with that many
 *                    variants per workgroup: one launch per step, each step
 *                    cut into chunks of 256 positions taken by separate
 *                    workgroups (DD_EINVAL when the schedule has more than
 *                    512 steps); any other value returns DD_EINVAL.
 *   dd_simulate_batch itself takes the few-variant path when the variants
 *   are fewer than 1,024, the schedule has at most 512 steps, and its steps
 *   hold more than about 4.4 rounds of 512 positions on average (where that
 *   path measured faster).
 * The results do not depend on the shape (Algorithm 1 per variant, Sec. 4.1);
 * only the number of workgroups and the kernel instance do.  For tuning, and
 * for checking every compiled instance.
 */
dd_status dd_simulate_batch_vs(const dd_graph *g, const dd_sched *sched, const dd_variants *var,
                               int64_t *d_finish, int64_t *d_start, int64_t *d_makespan,
                               int32_t variants_per_wg, void *stream);

/*
 * dd_set_lookback_polls -- how long a chunk of the few-variant path waits
 * for an earlier chunk (Sec. 4.1: the releases of one thread's run carried
 * across chunks).  A chunk reads the aggregate that each earlier chunk of its
 * run publishes; after `polls` unanswered reads it folds that chunk itself
 * from the inputs, which come from earlier launches, so no chunk ever depends
 * on another workgroup being resident.  The results do not depend on the
 * value.  polls < 0 restores the default (4,096); 0 makes every chunk fold
 * its predecessors itself (for tests of that fallback).  Applies to calls
 * made after it, process-wide.
 */
void dd_set_lookback_polls(int32_t polls);

/*
 * dd_simulate_batch_noalloc -- dd_simulate_batch for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, results and errors as
 * dd_simulate_batch; it always runs the one-workgroup-per-strip kernel with
 * the library's strip width (never the few-variant path, whose look-back
 * slots it would have to allocate), calls no hipMalloc, hipFree or other
 * allocating routine and records no events.
 *   Its working memory (round table, scan sums, per-position removal bits)
 *   lives in one array of 64 MiB per GPU inside the library, held until the
 *   process ends.  A batch needs about n*V/8 + 16*n_steps + 4*n/64 bytes of
 *   it (n*V up to about 5 * 10^8 task-variant pairs); a larger one returns
 *   DD_EINVAL with the size in dd_last_error() and launches nothing.
 *   Every call on one GPU uses that GPU's array: calls that overlap on one
 *   GPU (on different streams, or from several host threads) race and give
 *   wrong results.  The array keeps the last call's contents; nothing in it
 *   needs to start at zero.
 *   Handles used here on a stream other than their own are not tracked (no
 *   event is recorded): free them only after that stream's work is done.
 */
dd_status dd_simulate_batch_noalloc(const dd_graph *g, const dd_sched *sched, const dd_variants *var,
                                    int64_t *d_finish, int64_t *d_start, int64_t *d_makespan,
                                    void *stream);

/*
 * dd_runtime_breakdown -- where each variant's iteration time goes when the
 * CPU and the GPU overlap: the breakdown the paper uses to explain the AMP
 * speedups (Sec. 6.2, Fig. 6), computed by its own rules from a finished
 * dd_simulate_batch of the same graph and variants:
 *   total    = makespan;
 *   CPU-only = total - all GPU kernel runtime (the sum of the scaled
 *              durations of the kernels kept in the variant);
 *   GPU-only = the time the CPU is blocked on the GPU: for every call that
 *              waits for GPU work (synchronization, device-to-host copy), its
 *              start minus the moment its thread reached it (the release
 *              start + duration + gap of the previous task on the thread, 0
 *              for the first task);
 *   CPU+GPU parallel = total - CPU-only - GPU-only.
 *   role        uint8 [n], host or device: 1 = GPU kernel, 2 = CPU call that
 *               waits for GPU work, any other value = neither.
 *   d_finish    device int64 [n][V], d_makespan device int64 [V]: the outputs
 *               of dd_simulate_batch for (g, var), complete on `stream`.
 *   d_out       device int64 [V][4]: total, CPU-only, GPU-only, CPU+GPU
 *               parallel of each variant.
 * Asynchronous like dd_simulate_batch.  DD_EMISMATCH if var comes from
 * another graph.
 */
dd_status dd_runtime_breakdown(const dd_graph *g, const dd_variants *var, const uint8_t *role,
                               const int64_t *d_finish, const int64_t *d_makespan,
                               int64_t *d_out, void *stream);

/*
 * dd_simulate_policy -- simulate every variant with an overridden schedule()
 * (Sec. 4.4, "Schedule"): Algorithm 1 task by task, where schedule() picks
 * the next task from the frontier Q of ready tasks, kept in trace order
 * (ascending task id).  With time(x) = max(P[x's thread], x's start):
 *   DD_POLICY_EARLIEST  the first task of least time (the default rule);
 *   DD_POLICY_PRIORITY  P3's rule (the appendix's P3 model, its Schedule
 *                       function): scanning Q in order, a task of least time
 *                       is chosen, and a later task of equal time replaces
 *                       the choice when both are push/pull tasks (pp != 0)
 *                       and its priority is strictly higher.
 * On graphs whose threads are single chains every rule gives the result of
 * dd_simulate_batch.  Transformations as above (removed tasks run with zero
 * duration and gap); every variant's own edge classes apply, so one call
 * covers all variants of `var` without a schedule handle.
 *   pp, prio    uint8 [n] and int32 [n], host or device, read by
 *               DD_POLICY_PRIORITY (may be NULL for DD_POLICY_EARLIEST).
 *   d_finish    device int64 [n][V] (task-major, variant-minor), required
 *               unless n == 0.   d_start: the same or NULL.
 *   d_makespan  device int64 [V], required.
 * Limits: n < 2^22, n_threads <= 4096, in_ptr[n] + n < 2^31, and at most
 * 1024 tasks ready at once in any variant (DD_ELIMIT beyond, outputs
 * undefined).
 * Synchronous: returns when the simulation is done, with DD_ECYCLE if some
 * variant's active dependencies and thread chains contain a cycle.  Working
 * memory: 12 * n * V bytes of device memory for the call.
 */
#define DD_POLICY_EARLIEST 0
#define DD_POLICY_PRIORITY 1
dd_status dd_simulate_policy(const dd_graph *g, const dd_variants *var, int32_t policy,
                             const uint8_t *pp, const int32_t *prio,
                             int64_t *d_finish, int64_t *d_start, int64_t *d_makespan,
                             void *stream);

/*
 * dd_release_cache -- wait for all work on the current device, then return
 * every block of the library's device-memory cache for that device to the
 * device (hipFree).  Memory held by live handles is not touched.  For callers
 * that share the GPU with another allocator (e.g. torch) and need the space.
 */
dd_status dd_release_cache(void);

/* Step (level or phase) of every task: int32 [n], host or device pointer. */
dd_status dd_sched_task_steps(const dd_sched *sched, int32_t *steps_out, void *stream);

/*
 * dd_simulate_plan -- the launch shape dd_simulate_batch takes for these
 * handles, in the terms of dd_simulate_batch_vs: *variants_per_wg = 1, 2, 4,
 * 8 or 16 (one workgroup per strip of that many variants for the whole
 * schedule, one launch) or -1, -2, -4, -8 (the few-variant path, one launch per
 * step).  DD_EINVAL on a NULL argument.
 */
dd_status dd_simulate_plan(const dd_sched *sched, const dd_variants *var,
                           int32_t *variants_per_wg);

/* Schedule shape: steps, thread runs (segments), widest step, gather entries. */
dd_status dd_sched_info(const dd_sched *sched, int64_t *n_steps, int64_t *n_segments,
                        int64_t *max_step_width, int64_t *n_gathers);

void dd_graph_free(dd_graph *g);
void dd_sched_free(dd_sched *s);
void dd_variants_free(dd_variants *v);

const char *dd_status_str(dd_status s);
const char *dd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DD_H */
