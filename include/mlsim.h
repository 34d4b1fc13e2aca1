/*
 * mlsim.h -- C ABI of the batched dataflow replay library (libmlsim.so).
 *
 * The library replays one training iteration, given as a dataflow graph of
 * profiled ops, for many independent scenarios at once on one AMD Instinct
 * MI355X (gfx950).  It follows the simulation module of the paper
 * (Huang et al., "Simulating Performance of ML Systems with Offline
 * Profiling", Sec. 2, "Dataflow based simulation"):
 *   - ops are nodes, data/synchronisation dependencies are edges, and every op
 *     belongs to one device or communication link (a "resource");
 *   - every resource runs in parallel and keeps a job queue and its finish
 *     time; an op whose predecessors have all finished is ready and is queued
 *     on its resource; each resource serves its queue one op at a time,
 *     first-in-first-out by ready time (Sec. 4, future work, states the FIFO
 *     assumption);
 *   - the iteration time is the finish time of the last resource.
 * Points the paper leaves open are fixed as follows (the same for every
 * algorithm this library offers, and bit-identical between them):
 *   - equal ready times are served by lower priority value, then lower op id;
 *     every op finishing at time t is retired before anything starts at t;
 *   - sources are ready at t = 0, resources are free at t = 0, edges add no
 *     latency, an op never shares its resource (no preemption);
 *   - durations are int32 nanoseconds and must be >= 1; all times are exact
 *     integers; a time above INT32_MAX is reported, never wrapped.
 *
 * Conventions: every function returns an int status (SIM_OK = 0, or a
 * negative SIM_E_* code) unless stated.  "device" pointers are HIP device
 * (or managed) memory owned by the caller; "host" pointers are ordinary
 * memory.  Arrays of shape [n_ops][ld] are op-major: entry (v, s) is at
 * v * ld + s, so one op's values for consecutive scenarios are contiguous.
 *
 * Streams and graphs: a graph is read-only after creation, and calls on
 * different streams may share it and overlap in time.  Each graph owns a
 * few sets of scratch memory (allocated by sim_graph_create, never by a
 * call); a call takes one set for its kernels and records an event after
 * them, and a later call that takes the same set first makes its own stream
 * wait for that event, so no two calls use one set at once (on devices with
 * room for several sets, overlapping calls on different streams run
 * concurrently; otherwise they run one after the other).  Calls made while
 * their stream is being captured into a HIP graph use a set of their own
 * and record no event; replays of such captured graphs must not overlap one
 * another.
 * Streams are hipStream_t passed as void* (NULL = the null stream).
 */
#ifndef MLSIM_H
#define MLSIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* return codes */
enum {
  SIM_OK = 0,
  SIM_E_INVAL = -1, /* bad argument: NULL where an array is required, ld < n_scen, bad CSR pointers */
  SIM_E_RANGE = -2, /* an index out of range: successor id, op resource */
  SIM_E_CYCLE = -3, /* the graph has a cycle (including self loops) */
  SIM_E_NOMEM = -4, /* host or device allocation failed */
  SIM_E_HIP = -5,   /* a HIP runtime call failed (e.g. no GPU) */
  SIM_E_LIMIT = -6  /* the graph exceeds a size limit of this library */
};

/* per-scenario status bits (status[s]); a scenario with any bit set has
 * makespan[s] = -1 and unspecified finish values */
enum {
  SIM_ST_BAD_DUR = 1,  /* some duration < 1 */
  SIM_ST_BAD_RES = 2,  /* some placement >= n_res */
  SIM_ST_OVERFLOW = 4, /* a finish time exceeds INT32_MAX (only reported when
                          neither bit above is set) */
  SIM_ST_SHARE_LIMIT = 8, /* sim_run_batch_share: more than SIM_SHARE_MAX ops at
                             once on one shared resource */
  SIM_ST_INTERNAL = 16    /* sim_run_batch_share: a consistency check of the
                             library failed (a defect; please report) */
};

/* bandwidth sharing (sim_run_batch_share): most ops active at once on one
 * shared resource, and the service units a resource delivers per ns
 * (2^12 lcm(1..16), below 2^32: k active ops get exactly equal shares when k
 * divides it, every k <= 16 among them) */
#define SIM_SHARE_MAX 64
#define SIM_SHARE_UNIT 2952069120u

/* sim_run_batch flags & 3: which exact algorithm computes the replay (3 is
 * not a valid value) */
enum {
  SIM_ALGO_AUTO = 0,  /* library's choice (currently EVENT) */
  SIM_ALGO_EVENT = 1, /* event-driven list scheduling, one scenario per lane */
  SIM_ALGO_SWEEP = 2  /* level-synchronous conservative sweeps */
};

/* limits */
#define SIM_MAX_OPS (1 << 24)
#define SIM_MAX_RES 1024

typedef struct sim_graph sim_graph; /* opaque; immutable after creation */

/*
 * Build a graph (Sec. 2: the dataflow graph with each node's "device"
 * property; the paper's preprocessing module turns framework graphs into
 * this unified form).
 *   n_ops   number of ops, 0 <= n_ops <= SIM_MAX_OPS.
 *   n_res   number of resources, 1 <= n_res <= SIM_MAX_RES.
 *   succ_ptr host int64 [n_ops+1]: succ_ptr[0] = 0, nondecreasing.
 *   succ_idx host int32 [succ_ptr[n_ops]]: successor op ids in [0, n_ops);
 *            repeated edges are allowed and act as one edge.
 *   op_res  host int32 [n_ops]: resource of each op, in [0, n_res).
 *   prio    host int32 [n_ops] or NULL (NULL: prio[v] = v).  Lower values
 *           are served first among ops with equal ready time; ties in
 *           priority go to the lower op id.
 *   out     receives the graph.
 * Every host array is copied; the caller may free them on return.  The graph
 * owns its device copy and all scratch memory it needs (sized here, for any
 * number of scenarios).  Needs a HIP device (the current one); argument,
 * range and cycle errors are detected first, without touching the GPU.
 */
int sim_graph_create(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                     const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                     sim_graph **out);

/* Free a graph.  The caller must first synchronise every stream that used it. */
void sim_graph_destroy(sim_graph *g);

/*
 * Replay n_scen scenarios (Sec. 2's simulation loop, once per scenario).
 *   dur      device int32 [n_ops][ld_dur], ld_dur >= n_scen: duration (ns)
 *            of op v in scenario s at v * ld_dur + s.
 *   place    device uint16 [n_ops][ld_place] or NULL: if given, op v runs on
 *            resource place[v * ld_place + s] in scenario s instead of op_res[v].
 *   makespan device int32 [n_scen]: iteration time (the finish time of the
 *            last resource), or -1 if status[s] != 0.
 *   finish   device int32 [n_ops][ld_fin] or NULL: finish time of every op.
 *   status   device int32 [n_scen] or NULL: SIM_ST_* bits.
 *   flags    SIM_ALGO_* in bits 0-1; other bits must be 0.
 *   stream   hipStream_t (void*), NULL for the null stream.
 * Asynchronous on `stream`.  Argument errors return synchronously before
 * anything is enqueued.  No memory is allocated.  Calls on different streams
 * that share one graph may overlap (see "Streams and graphs" above).
 */
int sim_run_batch(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                  const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                  int64_t ld_fin, int32_t *status, uint32_t flags, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * sim_run_batch with the event algorithm, its per-block scratch taken from
 * one fixed array in the library's static device memory instead of the
 * graph's scratch sets.  The array holds SIM_NOALLOC_SCRATCH_BYTES per GPU
 * (the library looks up each device's copy once, when the first graph is
 * created on it, and every GPU the library runs on keeps it until the
 * process ends).  The call allocates nothing and clears the part of the
 * array it uses with a kernel before the replay.
 *   Arguments and outputs as sim_run_batch; flags SIM_ALGO_AUTO or
 *   SIM_ALGO_EVENT (others: SIM_E_INVAL).  Results equal sim_run_batch's.
 *   Returns SIM_E_LIMIT when one block's scratch (the graph's bound on ready
 *   ops, its joins and, for more resources than LDS holds, its resource
 *   times, per lane) exceeds the array; more scenarios only take more
 *   rounds of the persistent grid (fewer blocks run at once than in
 *   sim_run_batch when the array is smaller than the graph's sets).
 * Every call on one GPU shares that GPU's array and leaves its contents
 * behind: calls that overlap in time on one GPU (other streams, other
 * graphs, other threads) race and their results are undefined.  Calls on
 * one stream are ordered.  Asynchronous on `stream`.
 */
#define SIM_NOALLOC_SCRATCH_BYTES (128u << 20)
int sim_run_batch_noalloc(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                          const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                          int64_t ld_fin, int32_t *status, uint32_t flags, void *stream);

/*
 * The replay with a gap per resource.  The paper attributes part of its
 * simulator's remaining error to the idle time between consecutive ops on a
 * device, which its loop does not model (Sec. 3).  Here a resource that
 * finishes an op at time f cannot start its next op before f + gap[r]; its
 * first op is not delayed.  An op popped from the ready list therefore
 * starts at max(ready time, previous finish on its resource + gap[r]); the
 * queues stay first-in-first-out by ready time, with the same tie rules, and
 * the makespan is the largest finish time (a trailing gap does not count).
 *   gap  host int32 [n_res], every entry >= 0 (else SIM_E_INVAL); read
 *        before the call returns (its values travel to the graph's scratch
 *        memory in stream order as kernel arguments).
 * Other arguments and outputs as sim_run_batch (placement allowed; a finish
 * time above INT32_MAX sets SIM_ST_OVERFLOW); flags: SIM_ALGO_AUTO or
 * SIM_ALGO_EVENT (others return SIM_E_INVAL).  With every gap 0 the result
 * equals sim_run_batch.  Asynchronous on `stream`; no memory is allocated.
 */
int sim_run_batch_gap(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                      const uint16_t *place, int64_t ld_place, const int32_t *gap,
                      int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                      uint32_t flags, void *stream);

/*
 * The replay with a device model: a gap per resource (as sim_run_batch_gap)
 * and an output delay per resource.  The paper names memory copies, with
 * the gaps between ops, among the costs its loop leaves out (Sec. 3).  Here
 * the outputs of an op that finishes at f on resource r reach its
 * successors at f + delay[r] (a copy that does not occupy the resource: r
 * can start its next op at f, or f + gap[r]).  An op is ready when the
 * outputs of all its predecessors have arrived, and its queue order uses
 * that ready time.  The makespan stays the largest finish time (the delay
 * after the last op does not count).
 *   gap    host int32 [n_res] or NULL (no gaps), every entry >= 0.
 *   delay  host int32 [n_res] or NULL (no delays), every entry >= 0.
 *          A negative entry returns SIM_E_INVAL.  Both arrays are read
 *          before the call returns (their values travel to the graph's
 *          scratch memory in stream order as kernel arguments).
 * Other arguments, outputs and flags as sim_run_batch_gap; with both arrays
 * NULL, or all entries 0, the result equals sim_run_batch.  Asynchronous on
 * `stream`; no memory is allocated.
 */
int sim_run_batch_dev(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                      const uint16_t *place, int64_t ld_place, const int32_t *gap,
                      const int32_t *delay, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                      int32_t *status, uint32_t flags, void *stream);

/*
 * The replay with bandwidth sharing on chosen resources.  The paper leaves
 * concurrent transfers dividing one link's bandwidth to future work
 * (Sec. 4).  A resource with share[r] != 0 has no queue: every op that
 * becomes ready on it starts at once, and its active ops divide its rate
 * equally (processor sharing); an op's duration is its time when alone.
 * Time stays in integer ns: between two consecutive event times t1 < t2
 * each of the k active ops receives (t2 - t1) * floor(SIM_SHARE_UNIT / k)
 * service units (an exact equal share when k divides SIM_SHARE_UNIT); an
 * op needs dur * SIM_SHARE_UNIT units and finishes at the first integer ns
 * at which it has them.  At one time, finishes on shared
 * resources (lower resource first) come before ready ops, which keep the
 * (ready time, priority, id) order of sim_run_batch; other resources run
 * first in first out as there.  The makespan is the largest finish time.
 *   share  host uint8 [n_res] (nonzero: shared) or NULL (none shared, the
 *          result of sim_run_batch); read before the call returns.
 *   status SIM_ST_BAD_DUR, SIM_ST_OVERFLOW (a finish time above INT32_MAX),
 *          SIM_ST_SHARE_LIMIT (more than SIM_SHARE_MAX ops at once on one
 *          shared resource); a scenario's replay stops at the first
 *          overflow or limit event in time order.
 * dur, makespan, finish, ld_fin as sim_run_batch; no placement.  The
 * scratch memory of this replay is one set per graph, allocated by
 * sim_graph_create (up to about 8 GiB for large graphs, fewer block regions
 * when the device has less room); calls allocate nothing.  Calls on
 * different streams that share one graph are ordered one after the other
 * through that set's event; a call captured into a HIP graph uses the same
 * set, so its replays must not overlap any other sharing call on the graph.
 * Asynchronous on `stream`.
 */
int sim_run_batch_share(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                        const uint8_t *share, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                        int32_t *status, void *stream);

/*
 * Critical path per scenario: the longest path through the graph with
 * resources ignored, dist(v) = d(v) + max over predecessors of dist (0 if
 * none), cp_len[s] = max over v of dist(v); 0 for an empty graph, -1 if a
 * duration is < 1 or a path exceeds INT32_MAX.  It is the iteration time
 * with unlimited resources and the bound the paper's bottleneck analysis
 * starts from (Sec. 1).
 *   dur      device int32 [n_ops][ld_dur], ld_dur >= n_scen.
 *   cp_len   device int32 [n_scen].
 *   path_scen  -1, or a scenario whose path is returned: then path_ops (host
 *            int32, capacity path_cap) receives the path from its first op to
 *            its last and *path_len (host) its length (written even if larger
 *            than path_cap).  The last op is the lowest-id op of maximum dist;
 *            each step back goes to the lowest-id predecessor p with
 *            dist(p) = dist(v) - d(v).  With a path request the call
 *            synchronises `stream` before returning.
 * Otherwise asynchronous on `stream`; no memory is allocated.
 */
int sim_critical_path(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                      int32_t *cp_len, int64_t path_scen, int32_t *path_ops, int32_t path_cap,
                      int32_t *path_len, void *stream);

/* Static, human-readable text for a return code. */
const char *sim_strerror(int code);

/* Graph properties after compilation (host ints, any pointer may be NULL):
 * ops, resources, edges kept after removing duplicate and transitively
 * implied edges, ops with two or more predecessors, and the number of
 * distinct topological levels. */
int sim_graph_info(const sim_graph *g, int32_t *n_ops, int32_t *n_res, int64_t *n_edges,
                   int32_t *n_joins, int32_t *n_levels);

/*
 * Bottleneck attribution (Sec. 1: the simulator is used to find the
 * performance bottleneck).  Replays every scenario as sim_run_batch does
 * (same dur/place/makespan/status/finish arguments; finish and status are
 * required here) and additionally returns, per scenario s without status
 * bits:
 *   prev      device int32 [n_ops][ld_op] (required): the op that ran right
 *             before op v on its resource, -1 if none (same ld as finish);
 *   busy      device int32 [n_res][ld_res]: total duration of the ops
 *             resource r ran;
 *   chain     device int32 [n_res][ld_res]: time the binding chain spends on
 *             resource r; a scenario's entries sum to its makespan;
 *   chain_ops device int32 [n_scen]: ops on the binding chain.
 * The binding chain starts at the lowest-id op with the largest finish time
 * and walks back: from an op that starts at t > 0 to the lowest-id
 * predecessor that finished at t if one did (its input arrived last), else to
 * the op that ran before it on its resource (which finished at t: the op
 * waited for its resource); it ends at an op that starts at 0.  Scenarios
 * with status bits get busy = chain = 0 and chain_ops = -1.  path_scen,
 * path_ops, path_cap and path_len as in sim_critical_path, for the binding
 * chain (from its first op to its last; length 0 for a flagged scenario);
 * with a path request the call synchronises `stream`.  Otherwise
 * asynchronous; no memory is allocated.
 */
int sim_attribute(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                  const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *status,
                  int32_t *finish, int32_t *prev, int64_t ld_op, int32_t *busy, int32_t *chain,
                  int64_t ld_res, int32_t *chain_ops, int64_t path_scen, int32_t *path_ops,
                  int32_t path_cap, int32_t *path_len, void *stream);

/*
 * Static-order replay.  Sec. 2's devices each keep a queue of jobs; here
 * every device runs its ops in one order fixed in advance: the order in
 * which they appear in `order`.  An op starts when all its predecessors and
 * the op before it on its device have finished:
 *   finish(v) = d(v) + max(finish of v's predecessors,
 *                          finish of the previous op on res(v) in order, 0).
 * Given the order in which the event replay ran each device in a scenario,
 * it reproduces that scenario's finish times exactly.
 *
 * sim_static_create compiles the order against a graph (resources from the
 * graph's op_res):
 *   order  host int32 [n_ops]: a permutation of 0..n_ops-1 (copied).
 * Returns SIM_E_INVAL if order is NULL (n_ops > 0) or not a permutation,
 * SIM_E_CYCLE if the device orders contradict the dependencies (the DAG
 * plus each device's order has a cycle).  The result does not refer to g
 * after creation.  Allocates device memory on the current device.
 */
typedef struct sim_static sim_static; /* opaque; immutable after creation */
int sim_static_create(const sim_graph *g, const int32_t *order, sim_static **out);

/* Free a static-order replay.  The caller must first synchronise every
 * stream that used it. */
void sim_static_destroy(sim_static *st);

/*
 * Run the static-order replay for n_scen scenarios.  Arguments, outputs and
 * status bits as sim_run_batch without placement: makespan = max finish, or
 * -1 with SIM_ST_BAD_DUR (a duration < 1) or SIM_ST_OVERFLOW (a finish time
 * above INT32_MAX) in status; finish values of such scenarios are
 * unspecified.  Asynchronous on `stream`; no memory is allocated.  Calls on
 * different streams may share one object: when its value slots live in
 * global memory (one set, allocated by sim_static_create) a call waits for
 * the previous user of that set as described for graphs above.
 */
int sim_static_run(const sim_static *st, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                   int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                   void *stream);

/*
 * On-device scenario generation.  The paper's simulator exists to evaluate
 * many parallelisation strategies and configurations quickly (Sec. 1), and
 * its profiled op times vary by under 1 % of their mean (Sec. 3).  These
 * calls take a table of base durations per strategy knob instead of a
 * duration matrix and compute every duration inside the kernels:
 *   global scenario S = scen0 + s, knob k = (S / knob_block) mod n_knobs,
 *   b = base[k * n_ops + v];
 *   (x0, x1, x2, x3) = Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) of
 *       the counter (lo32 S, hi32 S, v, 0) under the key (lo32 seed, hi32 seed);
 *   U = the sum of the eight 16-bit halves of x0..x3, t = 2U - 524280;
 *   d(v, s) = b + floor((b * t * noise + 2^39) / 2^40)
 * in exact integer arithmetic, so every call, kernel and host reproduces the
 * same durations.  The relative noise has mean 0 and standard deviation
 * noise * 2 sqrt(2 (65536^2 - 1) / 3) / 2^40 (about noise * 9.7334e-8;
 * noise = 102739 gives 1 %); its shape is an 8-term Irwin-Hall sum (bounded,
 * nearly normal).  Durations then follow the sim_run_batch rules; a base
 * outside [1, SIM_GEN_BASE_MAX] yields d = 0, reported as SIM_ST_BAD_DUR.
 * Common arguments:
 *   base       device int32 [n_knobs][n_ops] (caller-owned, read only).
 *   n_knobs    >= 1; knob_block >= 1 (scenarios sharing a knob).
 *   noise      < SIM_GEN_NOISE_MAX (so that d >= b / 2 >= 1); 0: no noise.
 *   seed       the Philox key.
 *   scen0      >= 0: global index of scenario 0, so a sweep split over calls
 *              (or devices) generates the same scenarios as one call.
 * Any other value returns SIM_E_INVAL before anything is enqueued, as does
 * scen0 + n_scen > INT64_MAX.  Asynchronous on `stream`; no memory is
 * allocated.
 */
#define SIM_GEN_BASE_MAX (1 << 24)
#define SIM_GEN_NOISE_MAX (1u << 20)

/* Write the generated durations: dur device int32 [n_ops][ld_dur], ld_dur >= n_scen. */
int sim_generate(int32_t n_ops, int64_t n_scen, const int32_t *base, int32_t n_knobs,
                 int64_t knob_block, uint32_t noise, uint64_t seed, int64_t scen0, int32_t *dur,
                 int64_t ld_dur, void *stream);

/* sim_run_batch on generated durations, without placement; makespan, finish,
 * ld_fin, status and stream as there.  flags: SIM_ALGO_AUTO or SIM_ALGO_EVENT
 * (the event kernel; other values return SIM_E_INVAL). */
int sim_run_generated(const sim_graph *g, int64_t n_scen, const int32_t *base, int32_t n_knobs,
                      int64_t knob_block, uint32_t noise, uint64_t seed, int64_t scen0,
                      int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                      uint32_t flags, void *stream);

/* sim_critical_path on generated durations; cp_len, path_scen, path_ops,
 * path_cap, path_len and stream as there (a path request synchronises
 * `stream`). */
int sim_critical_path_generated(const sim_graph *g, int64_t n_scen, const int32_t *base,
                                int32_t n_knobs, int64_t knob_block, uint32_t noise, uint64_t seed,
                                int64_t scen0, int32_t *cp_len, int64_t path_scen, int32_t *path_ops,
                                int32_t path_cap, int32_t *path_len, void *stream);

/* sim_static_run on generated durations (the generation arguments above);
 * makespan, finish, ld_fin, status and stream as sim_static_run. */
int sim_static_run_generated(const sim_static *st, int64_t n_scen, const int32_t *base,
                             int32_t n_knobs, int64_t knob_block, uint32_t noise, uint64_t seed,
                             int64_t scen0, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                             int32_t *status, void *stream);

#ifdef __cplusplus
}
#endif
#endif
