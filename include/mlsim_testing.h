/*
 * mlsim_testing.h -- testing entry point of libmlsim.so (not needed to use
 * the library).
 *
 * The library picks, once per graph, where each kernel keeps its per-lane
 * state (LDS, registers or global scratch) and how many blocks its
 * persistent grids hold.  Every choice computes the same results; this call
 * pins a graph to one of them so that a test can check each variant against
 * the oracle.  No environment variable or other hidden state selects a
 * variant.
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
  SIM_TEST_RF_GLOBAL = 6      /* value 0/1: the event kernel's resource times in global scratch (1) */
};

/*
 * Pin graph g to a kernel variant (what = SIM_TEST_*, value as listed) and
 * plan its launches and scratch again (its scratch sets are freed and
 * allocated anew).  The call synchronises the device first; no other thread
 * may use g during it.  Returns SIM_OK, SIM_E_INVAL for an unknown `what` or
 * a value out of range, or the allocation's error.
 */
int sim_testing_replan(sim_graph *g, int32_t what, int32_t value);

#ifdef __cplusplus
}
#endif
#endif
