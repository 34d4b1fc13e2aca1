/*
 * mlsim_testing.h -- testing entry point of libmlsim.so (not needed to use
 * the library).
 *
 * The library picks, once per graph, where each kernel keeps its per-lane
 * state (LDS, registers or global scratch) and how many blocks its
 * persistent grids hold.  Every choice computes the same results;
 * sim_testing_replan pins a graph to one of them so that a test can check
 * each variant against the oracle.  No environment variable or other hidden
 * state selects a variant.  sim_testing_sweep_table returns the max-plus
 * sweep table built for a graph, for CPU tests of the table builder, and
 * sim_testing_join_slots the event replay's join state slots.
 */
#ifndef MLSIM_TESTING_H
#define MLSIM_TESTING_H

#include <stdint.h>

#include "mlsim.h"

#ifdef __cplusplus
extern "C" {
#endif

enum {
  SIM_TEST_AUTO = 0,          /* forget every pin below: the library's own choices */
  SIM_TEST_EV_LDS_GROUPS = 1, /* value 0..8: groups of the event heap's third level kept in LDS; -1: auto */
  /* 2: unused */
  SIM_TEST_EV_BLOCKS_CAP = 3, /* value >= 1: at most this many blocks in the event kernel's persistent
                                 grid; 0: no cap */
  SIM_TEST_EV_REG = 4,        /* value 0/1: the heap root's children in registers (where available);
                                 -1: auto (registers when the chip is full) */
  SIM_TEST_CP_GLOBAL = 5,     /* value 0/1: the max-plus sweeps' value slots in global scratch (1) even
                                 when LDS holds them (static-order replays created afterwards too) */
  SIM_TEST_RF_GLOBAL = 6,     /* value 0/1: the event kernel's resource times in global scratch (1) */
  SIM_TEST_SHARE_KEY_ID = 7   /* value 0/1: the sharing replay's ready-op key words hold only the op id
                                 (1), as for graphs whose ids and resources do not fit 32 bits together */
};

/*
 * Pin graph g to a kernel variant (what = SIM_TEST_*, value as listed) and
 * plan its launches and scratch again (its scratch sets are freed and
 * allocated anew).  The call synchronises the device first; no other thread
 * may use g during it.  Returns SIM_OK, SIM_E_INVAL for an unknown `what` or
 * a value out of range, or the allocation's error.
 */
int sim_testing_replan(sim_graph *g, int32_t what, int32_t value);

/*
 * The max-plus sweep table the library builds, on the host only (no device
 * is used), so that a test can evaluate it on the CPU and compare the result
 * with an independent replay.  The graph arguments are those of
 * sim_graph_create.  order NULL: the critical-path table (sim_critical_path);
 * otherwise a permutation of the op ids whose restriction to each resource
 * is that resource's run order: the table of sim_static_create.
 * Outputs (host): *n_rec records in sweep order, each 8 int32 in rec
 * [rec_cap][8]: {row, slot, npred, pbeg, p0, p1, p2, p3} -- row: the op
 * (its dist is its finish time or path length), -1 for a barrier record
 * (duration 0); slot: the value slot receiving the record's dist; the
 * predecessor slots are p0..p(npred-1) when npred <= 4, else plist[pbeg ..
 * pbeg + npred); unused p entries name slot *slots - 2, which holds 0; a
 * record whose value nothing reads writes slot *slots - 1.  *plist_len
 * entries go to plist [plist_cap].  Returns SIM_OK; the argument errors of
 * sim_graph_create and sim_static_create (SIM_E_INVAL, SIM_E_RANGE,
 * SIM_E_CYCLE, SIM_E_LIMIT); or SIM_E_LIMIT when rec_cap or plist_cap is too
 * small, after writing *n_rec and *plist_len.
 */
int sim_testing_sweep_table(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                            const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                            const int32_t *order, int32_t *n_rec, int32_t *slots, int32_t *rec,
                            int64_t rec_cap, int32_t *plist, int64_t plist_cap, int64_t *plist_len);

/*
 * The join state slots of the event replay (sim_run_batch and the calls
 * built on it), on the host only.  An op whose predecessors, after removing
 * edges implied by longer paths, number two or more waits on a join: a
 * {predecessors finished, latest finish} word per lane, which the replay
 * updates when each of those predecessors finishes and clears when the last
 * one does.  Ops with the same predecessor set share one join.  Joins whose
 * words are never needed at the same time in any scenario may share a slot
 * (the replay's scratch then holds fewer words).  The graph arguments are
 * those of sim_graph_create.  Outputs (host): slot_of [n_ops]: the slot of
 * the join each op waits on, -1 for an op without one; *n_slots: the number
 * of slots.  Returns SIM_OK or the argument errors of sim_graph_create.
 */
int sim_testing_join_slots(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                           const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                           int32_t *slot_of, int32_t *n_slots);

#ifdef __cplusplus
}
#endif
#endif
