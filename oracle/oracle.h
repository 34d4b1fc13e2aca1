/*
 * CPU oracle for the batched dataflow replay -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow discrete-event simulator written from the paper's
 * description of its simulation module (Sec. 2, "Dataflow based
 * simulation"): every device or link runs in parallel and keeps a job queue
 * and its finish time; ready nodes are queued on their device; a finished
 * op decrements its successors' dependency counters and a counter reaching
 * zero makes the successor ready; the iteration time is the finish time of
 * the last device.  It is used only by tests and by the benchmark's CPU
 * baseline; nothing in the library calls it, links it or includes this
 * header.
 *
 * Readings of points the paper leaves open (listed in the design notes):
 *  - each device serves its queue first-in-first-out by ready time, one op
 *    at a time, without preemption; equal ready times are served by lower
 *    priority value, then lower op id;
 *  - all ops that finish at time t are applied before anything starts at t;
 *  - sources are ready at t = 0, every device is free at t = 0, edges add no
 *    latency, durations are integer nanoseconds >= 1;
 *  - a finish time above INT32_MAX is reported as an overflow, never wrapped.
 *
 * All functions take host pointers.  Graphs are given as successor CSR;
 * repeated edges are allowed and behave like a single edge.
 */
#ifndef MLSIM_ORACLE_H
#define MLSIM_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* return codes (same numbering as the library's, by interface contract) */
#define ORC_OK 0
#define ORC_E_INVAL (-1)
#define ORC_E_RANGE (-2)
#define ORC_E_CYCLE (-3)
#define ORC_E_NOMEM (-4)

/* per-scenario status bits */
#define ORC_ST_BAD_DUR 1
#define ORC_ST_BAD_RES 2
#define ORC_ST_OVERFLOW 4
#define ORC_ST_SHARE_LIMIT 8 /* more than ORC_SHARE_MAX ops at once on a shared device */

/* bandwidth sharing: concurrent ops per shared device, and the service units
 * a device delivers per ns (2^12 lcm(1..16), below 2^32: k active ops get
 * exactly equal shares whenever k divides it, every k <= 16 among them) */
#define ORC_SHARE_MAX 64
#define ORC_SHARE_UNIT 2952069120u

/*
 * Replay every scenario s in [0, n_scen).
 *   succ_ptr [n_ops+1], succ_idx [succ_ptr[n_ops]]: successor CSR.
 *   op_res   [n_ops]: resource of each op, in [0, n_res).
 *   prio     [n_ops] or NULL (NULL means prio[v] = v).
 *   dur      [n_ops][ld_dur]: duration of op v in scenario s is dur[v*ld_dur+s].
 *   place    [n_ops][ld_place] or NULL: if given, resource of v in s is
 *            place[v*ld_place+s] instead of op_res[v].
 * Outputs: makespan[s]; finish[v*ld_fin+s] if finish != NULL; status[s] if
 * status != NULL.  A scenario with a bad duration (< 1), a bad placement or
 * an overflow gets its status bits and makespan -1 (its finish values are
 * then unspecified).  n_threads <= 0 means 1.
 */
int oracle_run_batch(int32_t n_ops, int32_t n_res,
                     const int64_t *succ_ptr, const int32_t *succ_idx,
                     const int32_t *op_res, const int32_t *prio,
                     int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                     const uint16_t *place, int64_t ld_place,
                     int32_t *makespan, int32_t *finish, int64_t ld_fin,
                     int32_t *status, int32_t n_threads);

/*
 * The replay with a gap per device (the paper names the idle time between
 * consecutive ops on a device as a source of the simulator's residual error,
 * Sec. 3): after a device finishes an op it cannot start its next op for
 * gap[r] ns, so an op popped from the ready list starts at
 *   max(ready time, finish of the device's previous op + gap[r]),
 * or at its ready time if it is the device's first op.  Queues stay
 * first-in-first-out by ready time; the makespan is still the largest finish
 * time (a trailing gap does not count).  gap: [n_res] with every entry >= 0
 * (else ORC_E_INVAL), or NULL for no gaps (oracle_run_batch).  Everything
 * else as oracle_run_batch.
 */
int oracle_run_batch_gap(int32_t n_ops, int32_t n_res,
                         const int64_t *succ_ptr, const int32_t *succ_idx,
                         const int32_t *op_res, const int32_t *prio, const int32_t *gap,
                         int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                         const uint16_t *place, int64_t ld_place,
                         int32_t *makespan, int32_t *finish, int64_t ld_fin,
                         int32_t *status, int32_t n_threads);

/*
 * The replay with gaps and output delays per device.  The paper lists the
 * memcpy time around ops among its simulator's unmodelled overheads
 * (Sec. 3); here an op on device r hands its outputs to its successors
 * delay[r] ns after it finishes (the device itself is free at its finish,
 * plus its gap), so a successor's ready time is the largest
 * finish + delay[device] over its predecessors.  gap and delay: [n_res]
 * with entries >= 0 (else ORC_E_INVAL), each may be NULL (zeros).  The
 * makespan is the largest finish time.  Everything else as
 * oracle_run_batch.
 */
int oracle_run_batch_dev(int32_t n_ops, int32_t n_res,
                         const int64_t *succ_ptr, const int32_t *succ_idx,
                         const int32_t *op_res, const int32_t *prio, const int32_t *gap,
                         const int32_t *delay, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                         const uint16_t *place, int64_t ld_place,
                         int32_t *makespan, int32_t *finish, int64_t ld_fin,
                         int32_t *status, int32_t n_threads);

/*
 * The replay with bandwidth sharing on some devices.  The paper leaves
 * concurrent transfers dividing one link's bandwidth to future work
 * (Sec. 4).  A device with share[r] != 0 has no queue: every op that becomes
 * ready on it starts at once, and the ops active on it divide its rate
 * equally (processor sharing), an op's duration being its time when alone.
 * Time is kept in integer ns: between two consecutive event times t1 < t2
 * every active op receives (t2 - t1) * floor(ORC_SHARE_UNIT / k) service
 * units, k being the number of active ops (an exact equal share when k
 * divides ORC_SHARE_UNIT; otherwise less than k of ORC_SHARE_UNIT units per
 * ns go unused); an op needs dur * ORC_SHARE_UNIT units and finishes at the
 * first integer ns at which it has them.  Events at one time
 * are taken in this order: ops finishing on shared devices (lower device
 * first), then ready ops in (ready time, priority, id) order.  More than
 * ORC_SHARE_MAX ops at once on one shared device set ORC_ST_SHARE_LIMIT;
 * the replay of that scenario stops at the first such event or overflow.
 * Devices with share[r] == 0 behave as in oracle_run_batch.  share: [n_res]
 * or NULL (no shared devices).  No placement.
 */
int oracle_run_batch_share(int32_t n_ops, int32_t n_res,
                           const int64_t *succ_ptr, const int32_t *succ_idx,
                           const int32_t *op_res, const int32_t *prio, const uint8_t *share,
                           int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                           int32_t *makespan, int32_t *finish, int64_t ld_fin,
                           int32_t *status, int32_t n_threads);

/*
 * Longest path through the DAG, resources ignored: dist(v) = d(v) + max over
 * predecessors p of dist(p) (0 without predecessors); cp_len[s] = max_v
 * dist(v), 0 for an empty graph, -1 if a duration is < 1 or a path exceeds
 * INT32_MAX.  If path_scen >= 0, the path of that scenario is written to
 * path_ops (host, capacity path_cap) from its first op to its last, and its
 * length to *path_len (the length is written even if it exceeds path_cap):
 * the last op is the lowest-id op of maximum dist; each step back goes to
 * the lowest-id predecessor p with dist(p) = dist(v) - d(v).
 */
int oracle_critical_path(int32_t n_ops,
                         const int64_t *succ_ptr, const int32_t *succ_idx,
                         int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                         int32_t *cp_len, int64_t path_scen,
                         int32_t *path_ops, int32_t path_cap, int32_t *path_len,
                         int32_t n_threads);

/*
 * Static-order replay: every device runs its ops in the order they appear in
 * order[] (a permutation of 0..n_ops-1); an op starts when all its
 * predecessors and the previous op on its device (in that order) have
 * finished: finish(v) = d(v) + max(those finish times, 0).  Outputs and
 * status bits as oracle_run_batch (no placement: devices come from op_res).
 * Returns ORC_E_INVAL if order is not a permutation and ORC_E_CYCLE if the
 * device orders contradict the dependencies.
 */
int oracle_static_run(int32_t n_ops, int32_t n_res,
                      const int64_t *succ_ptr, const int32_t *succ_idx,
                      const int32_t *op_res, const int32_t *order,
                      int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                      int32_t *makespan, int32_t *finish, int64_t ld_fin,
                      int32_t *status, int32_t n_threads);

/*
 * Bottleneck attribution of the replay (same inputs as oracle_run_batch;
 * makespan and status as there).  Per scenario without status bits:
 *   busy[r*ld_res+s]   total duration of the ops device r ran;
 *   chain[r*ld_res+s]  time the binding chain spends on device r (the
 *                      entries of a scenario sum to its makespan);
 *   chain_ops[s]       ops on the binding chain (0 for an empty graph).
 * The binding chain starts at the lowest-id op of largest finish time; from
 * an op v starting at t > 0 it steps to the lowest-id predecessor finishing
 * at t if there is one, else to the op that ran before v on its device (it
 * finished at t); it ends at an op starting at 0.  Scenarios with status
 * bits get busy = chain = 0 and chain_ops = -1.  If path_scen >= 0 the chain
 * of that scenario is written to path_ops from its first op to its last and
 * its length to *path_len (0 for a flagged scenario).
 */
int oracle_attribute(int32_t n_ops, int32_t n_res,
                     const int64_t *succ_ptr, const int32_t *succ_idx,
                     const int32_t *op_res, const int32_t *prio,
                     int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                     const uint16_t *place, int64_t ld_place,
                     int32_t *makespan, int32_t *status,
                     int32_t *busy, int32_t *chain, int64_t ld_res,
                     int32_t *chain_ops, int64_t path_scen, int32_t *path_ops,
                     int32_t path_cap, int32_t *path_len, int32_t n_threads);

/*
 * Counter-based generators (Salmon et al., SC'11): Philox4x32-10 and
 * Philox4x64-10 applied to one counter block under one key.
 */
void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
void oracle_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);

/*
 * Scenario generation: durations of a strategy-knob grid with per-op
 * counter-based noise (the paper's motivation: many strategies and
 * configurations evaluated by simulation, Sec. 1; op times vary by under
 * 1 % of their mean, Sec. 3).  For op v and scenario s (global index
 * S = scen0 + s):
 *   knob k = (S / knob_block) mod n_knobs, b = base[k * n_ops + v];
 *   (x0..x3) = Philox4x32-10(counter (lo32 S, hi32 S, v, 0),
 *                            key (lo32 seed, hi32 seed));
 *   U = sum of the eight 16-bit halves of x0..x3, t = 2U - 524280;
 *   dur[v * ld_dur + s] = b + floor((b * t * noise + 2^39) / 2^40)
 * in exact 64-bit integer arithmetic; a base outside [1, 2^24] yields 0 (an
 * invalid duration).  noise must be below 2^20; the relative noise has
 * standard deviation noise * 2 sqrt(2 (65536^2 - 1) / 3) / 2^40, about
 * noise * 9.73e-8.  Returns ORC_E_INVAL for n_knobs < 1, knob_block < 1,
 * scen0 < 0, noise >= 2^20 or ld_dur < n_scen.
 */
int oracle_generate(int32_t n_ops, int64_t n_scen, const int32_t *base, int32_t n_knobs,
                    int64_t knob_block, uint32_t noise, uint64_t seed, int64_t scen0,
                    int32_t *dur, int64_t ld_dur, int32_t n_threads);

#ifdef __cplusplus
}
#endif
#endif
