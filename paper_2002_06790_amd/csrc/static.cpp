// Static-order replay: compile a fixed per-device run order against a graph
// into a max-plus sweep table (the DAG's predecessors plus each op's previous
// op on its device), and run it with the critical path's sweep kernel.
#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "sim.hpp"

using namespace mlsim;

struct sim_static {
  int32_t n_ops;
  int device;
  MpTable tab;      // device view of the records and long predecessor lists
  int mode;         // where the sweep's value slots live
  int blocks;       // persistent grid
  int gen_blocks;   // persistent grid with generated durations
  size_t lds;       // LDS bytes per block
  void *dev_mem;    // records and predecessor lists
  // global value slots when they do not fit LDS: one set, taken by each call
  // for its launch (calls on other streams wait for it)
  mutable ScratchPool slots;
  bool global_slots;
};

namespace {

constexpr size_t kSlotsLdsMax = 32 * 1024;
constexpr size_t kSlotsScratchBudget = 1ull << 30;

}  // namespace

namespace mlsim {

int static_table(int32_t n, const std::vector<int32_t> &orig_of, const std::vector<int32_t> &pred_ptr,
                 const std::vector<int32_t> &pred_c, const std::vector<int32_t> &res, const int32_t *order,
                 std::vector<CpRec> &rec, std::vector<int32_t> &plist, int32_t &slots, int32_t &n_sweep) {
  if (n > 0 && !order) return SIM_E_INVAL;
  // the order names every op once
  std::vector<char> seen(n, 0);
  for (int32_t k = 0; k < n; ++k) {
    const int32_t v = order[k];
    if (v < 0 || v >= n || seen[v]) return SIM_E_INVAL;
    seen[v] = 1;
  }
  // predecessors by caller id: the compiled DAG's (duplicates and implied
  // edges removed: an implied predecessor finishes before the one implying
  // it) and the previous op on the device in the given order
  std::vector<std::vector<int32_t>> pred(n), succ(n);
  for (int32_t c = 0; c < n; ++c) {
    const int32_t v = orig_of[c];
    for (int32_t k = pred_ptr[c]; k < pred_ptr[c + 1]; ++k) pred[v].push_back(orig_of[pred_c[k]]);
  }
  // extra[v]: the device predecessor when it is not already a DAG
  // predecessor (the sweep table compares predecessor sets without it);
  // pos[v]: v's place in the given order, which the sweep order prefers
  // among equally good choices
  std::vector<int32_t> last, extra(n, -1);
  std::vector<int64_t> pos(n);
  for (int32_t k = 0; k < n; ++k) {
    const int32_t v = order[k], r = res[v];
    if (r >= (int32_t)last.size()) last.resize(r + 1, -1);
    pos[v] = k;
    if (last[r] >= 0 && std::find(pred[v].begin(), pred[v].end(), last[r]) == pred[v].end()) {
      pred[v].push_back(last[r]);
      extra[v] = last[r];
    }
    last[r] = v;
  }
  for (int32_t v = 0; v < n; ++v) {
    std::sort(pred[v].begin(), pred[v].end());
    for (int32_t p : pred[v]) succ[p].push_back(v);
  }
  std::vector<int32_t> rows(n), sweep_order;
  for (int32_t v = 0; v < n; ++v) rows[v] = v;
  if (!build_maxplus(n, succ, pred, extra, pos, rows, rec, plist, slots, sweep_order, n_sweep)) return SIM_E_CYCLE;
  return SIM_OK;
}

}  // namespace mlsim

extern "C" int sim_static_create(const sim_graph *g, const int32_t *order, sim_static **out) {
  if (!out) return SIM_E_INVAL;
  *out = nullptr;
  if (!g) return SIM_E_INVAL;
  const int32_t n = g->n_ops;
  std::vector<CpRec> rec;
  std::vector<int32_t> plist;
  int32_t slots = 0, n_sweep = 0;
  try {
    if (int rc = static_table(n, g->h_orig_of, g->h_pred_ptr, g->h_pred, g->h_res, order, rec, plist, slots, n_sweep))
      return rc;
  } catch (const std::bad_alloc &) {
    return SIM_E_NOMEM;
  }

  sim_static *st = new (std::nothrow) sim_static();
  if (!st) return SIM_E_NOMEM;
  st->n_ops = n;
  st->dev_mem = nullptr;
  if (hipGetDevice(&st->device) != hipSuccess) {
    delete st;
    return SIM_E_HIP;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, st->device) != hipSuccess) {
    delete st;
    return SIM_E_HIP;
  }
  const size_t rec_bytes = rec.size() * sizeof(CpRec), pl_bytes = plist.size() * 4;
  const size_t pl_off = (rec_bytes + 255) & ~size_t(255);
  if (hipMalloc(&st->dev_mem, pl_off + pl_bytes) != hipSuccess) {
    delete st;
    return SIM_E_NOMEM;
  }
  char *base = (char *)st->dev_mem;
  if (hipMemcpy(base, rec.data(), rec_bytes, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(base + pl_off, plist.data(), pl_bytes, hipMemcpyHostToDevice) != hipSuccess) {
    sim_static_destroy(st);
    return SIM_E_HIP;
  }
  st->tab = MpTable{n_sweep, slots, (const CpRec *)base, (const int32_t *)(base + pl_off), n_sweep > n};
  // value slots in LDS when they fit, else in global scratch for the grid
  const size_t slot_bytes = (size_t)slots * kWave * 4;
  st->mode = slot_bytes <= kSlotsLdsMax && !g->var.cp_global ? kCpSlotsLds : kCpSlotsGlobal;
  st->lds = st->mode == kCpSlotsLds ? slot_bytes : 0;
  int blocks = maxplus_occupancy(st->mode, true, st->lds, prop.multiProcessorCount, false, st->tab.bar != 0);
  if (blocks < 0) {
    sim_static_destroy(st);
    return SIM_E_HIP;
  }
  if (st->mode == kCpSlotsGlobal) {
    blocks = (int)std::min<size_t>((size_t)blocks, std::max<size_t>(1, kSlotsScratchBudget / slot_bytes));
    auto clear = [](void *ctx, char *b) -> int {
      return hipMemset(b, 0, *(size_t *)ctx) == hipSuccess ? SIM_OK : SIM_E_HIP;
    };
    size_t bytes = slot_bytes * (size_t)blocks;
    st->global_slots = true;
    if (int rc = st->slots.init(bytes, 1, false, clear, &bytes)) {
      sim_static_destroy(st);
      return rc;
    }
  }
  st->blocks = std::max(1, blocks);
  const int gen_blocks = maxplus_occupancy(st->mode, true, st->lds, prop.multiProcessorCount, true, st->tab.bar != 0);
  if (gen_blocks < 0) {
    sim_static_destroy(st);
    return SIM_E_HIP;
  }
  st->gen_blocks = std::max(1, std::min(gen_blocks, st->blocks));  // within the slot scratch
  *out = st;
  return SIM_OK;
}

extern "C" void sim_static_destroy(sim_static *st) {
  if (!st) return;
  if (st->dev_mem) (void)hipFree(st->dev_mem);
  st->slots.destroy();
  delete st;
}

extern "C" int sim_static_run(const sim_static *st, int64_t n_scen, const int32_t *dur,
                              int64_t ld_dur, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                              int32_t *status, void *stream) {
  if (!st || n_scen < 0) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (st->n_ops > 0 && (!dur || ld_dur < n_scen)) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  if (st->n_ops == 0) {
    // no ops: every iteration takes 0 ns
    if (launch_zero(makespan, n_scen, n_scen, 1, s) != SIM_OK) return SIM_E_HIP;
    if (status && launch_zero(status, n_scen, n_scen, 1, s) != SIM_OK) return SIM_E_HIP;
    return SIM_OK;
  }
  if (!st->global_slots)
    return launch_maxplus(st->tab, st->mode, st->blocks, st->lds, n_scen, dur, ld_dur, makespan, status,
                          finish, ld_fin, nullptr, 0, nullptr, s);
  Lease lease(st->slots, s);
  if (lease.rc()) return lease.rc();
  return launch_maxplus(st->tab, st->mode, st->blocks, st->lds, n_scen, dur, ld_dur, makespan, status,
                        finish, ld_fin, nullptr, 0, (uint32_t *)lease.base(), s);
}

extern "C" int sim_static_run_generated(const sim_static *st, int64_t n_scen, const int32_t *base,
                                        int32_t n_knobs, int64_t knob_block, uint32_t noise, uint64_t seed,
                                        int64_t scen0, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                                        int32_t *status, void *stream) {
  if (!st || n_scen < 0) return SIM_E_INVAL;
  DurGen gen;
  if (int rc = make_gen(st->n_ops, n_scen, base, n_knobs, knob_block, noise, seed, scen0, gen)) return rc;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  if (st->n_ops == 0) {
    if (launch_zero(makespan, n_scen, n_scen, 1, s) != SIM_OK) return SIM_E_HIP;
    if (status && launch_zero(status, n_scen, n_scen, 1, s) != SIM_OK) return SIM_E_HIP;
    return SIM_OK;
  }
  if (!st->global_slots)
    return launch_maxplus(st->tab, st->mode, st->gen_blocks, st->lds, n_scen, nullptr, 0, makespan, status,
                          finish, ld_fin, nullptr, 0, nullptr, s, &gen);
  Lease lease(st->slots, s);
  if (lease.rc()) return lease.rc();
  return launch_maxplus(st->tab, st->mode, st->gen_blocks, st->lds, n_scen, nullptr, 0, makespan, status,
                        finish, ld_fin, nullptr, 0, (uint32_t *)lease.base(), s, &gen);
}
