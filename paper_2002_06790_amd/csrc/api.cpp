// C ABI entry points that run the kernels: argument checks, dispatch, and the
// host-side walk back along one scenario's critical path.
#include <algorithm>
#include <vector>

#include "sim.hpp"

using namespace mlsim;

namespace {

bool bad_matrix(const void *p, int64_t ld, int64_t n_scen, int32_t n_ops) {
  return n_ops > 0 && n_scen > 0 && (!p || ld < n_scen);
}

}  // namespace

extern "C" int sim_run_batch(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                             const uint16_t *place, int64_t ld_place, int32_t *makespan,
                             int32_t *finish, int64_t ld_fin, int32_t *status, uint32_t flags,
                             void *stream) {
  if (!g || n_scen < 0 || (flags & ~3u)) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (bad_matrix(dur, ld_dur, n_scen, g->n_ops)) return SIM_E_INVAL;
  if (place && ld_place < n_scen) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  if (g->n_ops == 0) {
    // no ops: every iteration takes 0 ns
    if (hipMemsetAsync(makespan, 0, (size_t)n_scen * 4, st) != hipSuccess) return SIM_E_HIP;
    if (status && hipMemsetAsync(status, 0, (size_t)n_scen * 4, st) != hipSuccess) return SIM_E_HIP;
    return SIM_OK;
  }
  const uint32_t algo = flags & 3u;
  if (algo == SIM_ALGO_SWEEP)
    return launch_sweep(g, n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin, status, st);
  // the lockstep walk needs one resource map for every scenario
  if (algo == SIM_ALGO_WALK && !place && walk_eligible(g))
    return launch_walk(g, n_scen, dur, ld_dur, makespan, finish, ld_fin, status, st);
  return launch_event(g, n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin, status,
                      st);
}

extern "C" int sim_critical_path(const sim_graph *g, int64_t n_scen, const int32_t *dur,
                                 int64_t ld_dur, int32_t *cp_len, int64_t path_scen,
                                 int32_t *path_ops, int32_t path_cap, int32_t *path_len,
                                 void *stream) {
  if (!g || n_scen < 0) return SIM_E_INVAL;
  if (path_scen >= n_scen || path_scen < -1) return SIM_E_INVAL;
  if (path_scen >= 0 && (!path_len || (path_cap > 0 && !path_ops) || path_cap < 0)) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!cp_len || bad_matrix(dur, ld_dur, n_scen, g->n_ops)) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  const int32_t n = g->n_ops;
  if (n == 0) {
    if (hipMemsetAsync(cp_len, 0, (size_t)n_scen * 4, st) != hipSuccess) return SIM_E_HIP;
    if (path_scen >= 0) *path_len = 0;
    return SIM_OK;
  }
  int32_t *dist_dev = path_scen >= 0 ? (int32_t *)((char *)g->scratch + g->scratch_dist_off) : nullptr;
  int rc = launch_cp(g, n_scen, dur, ld_dur, cp_len, dist_dev, path_scen, st);
  if (rc || path_scen < 0) return rc;

  // Walk back from the lowest-id op of maximum dist, each time to the
  // lowest-id predecessor p with dist(p) = dist(v) - d(v).
  std::vector<int32_t> dist(n), d(n);
  int32_t cp_s = 0;
  if (hipMemcpyAsync(dist.data(), dist_dev, (size_t)n * 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpy2DAsync(d.data(), 4, dur + path_scen, (size_t)ld_dur * 4, 4, n, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(&cp_s, cp_len + path_scen, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return SIM_E_HIP;
  if (cp_s < 0) {
    *path_len = 0;
    return SIM_OK;
  }
  std::vector<int32_t> comp(n);
  for (int32_t c = 0; c < n; ++c) comp[g->h_orig_of[c]] = c;
  int32_t v = -1;
  for (int32_t o = 0; o < n; ++o)
    if (dist[o] == cp_s) {
      v = o;
      break;
    }
  std::vector<int32_t> rev;
  while (v >= 0) {
    rev.push_back(v);
    const int32_t want = dist[v] - d[v];
    if (want == 0) break;
    int32_t nxt = -1;
    const int32_t c = comp[v];
    for (int32_t k = g->h_pred_ptr[c]; k < g->h_pred_ptr[c + 1]; ++k) {
      const int32_t p = g->h_orig_of[g->h_pred[k]];
      if (dist[p] == want && (nxt < 0 || p < nxt)) nxt = p;
    }
    v = nxt;
  }
  *path_len = (int32_t)rev.size();
  for (int32_t k = 0; k < (int32_t)rev.size() && k < path_cap; ++k) path_ops[k] = rev[rev.size() - 1 - k];
  return SIM_OK;
}
