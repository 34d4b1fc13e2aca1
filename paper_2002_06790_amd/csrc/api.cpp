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

// Walk back from the lowest-id op of maximum dist, each time to the
// lowest-id predecessor p with dist(p) = dist(v) - d(v); the path from its
// first op to its last goes to path_ops (up to path_cap), its length to
// *path_len.
void walk_critical_path(const sim_graph *g, const std::vector<int32_t> &dist, const std::vector<int32_t> &d,
                        int32_t cp_s, int32_t *path_ops, int32_t path_cap, int32_t *path_len) {
  const int32_t n = g->n_ops;
  if (cp_s < 0) {
    *path_len = 0;
    return;
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
}

}  // namespace

namespace mlsim {
int make_gen(int32_t n_ops, int64_t n_scen, const int32_t *base, int32_t n_knobs, int64_t knob_block,
             uint32_t noise, uint64_t seed, int64_t scen0, DurGen &gen) {
  if (n_knobs < 1 || knob_block < 1 || scen0 < 0 || noise >= kGenNoiseMax) return SIM_E_INVAL;
  if (n_scen > INT64_MAX - scen0) return SIM_E_INVAL;
  if (n_ops > 0 && !base) return SIM_E_INVAL;
  if ((int64_t)n_knobs * n_ops > INT64_MAX / 4) return SIM_E_INVAL;
  gen = DurGen{base, n_ops, n_knobs, knob_block, scen0, noise, (uint32_t)seed, (uint32_t)(seed >> 32)};
  return SIM_OK;
}
}  // namespace mlsim

extern "C" int sim_run_batch(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                             const uint16_t *place, int64_t ld_place, int32_t *makespan,
                             int32_t *finish, int64_t ld_fin, int32_t *status, uint32_t flags,
                             void *stream) {
  if (!g || n_scen < 0 || (flags & ~3u) || (flags & 3u) == 3u) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (bad_matrix(dur, ld_dur, n_scen, g->n_ops)) return SIM_E_INVAL;
  if (place && ld_place < n_scen) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  if (g->n_ops == 0) {
    // no ops: every iteration takes 0 ns
    if (launch_zero(makespan, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    if (status && launch_zero(status, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    return SIM_OK;
  }
  const uint32_t algo = flags & 3u;
  if (algo == 3u) return SIM_E_INVAL;
  if (algo == SIM_ALGO_SWEEP) {
    Lease lease(g->sweep_pool, st);
    if (lease.rc()) return lease.rc();
    return launch_sweep(g, lease.base(), n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin,
                        status, st);
  }
  Lease lease(g->pool, st);
  if (lease.rc()) return lease.rc();
  return launch_event(g, lease.base(), n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin,
                      status, st);
}

extern "C" int sim_run_batch_noalloc(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                                     const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                                     int64_t ld_fin, int32_t *status, uint32_t flags, void *stream) {
  if (!g || n_scen < 0 || (flags != SIM_ALGO_AUTO && flags != SIM_ALGO_EVENT)) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (bad_matrix(dur, ld_dur, n_scen, g->n_ops)) return SIM_E_INVAL;
  if (place && ld_place < n_scen) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  if (g->n_ops == 0) {
    if (launch_zero(makespan, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    if (status && launch_zero(status, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    return SIM_OK;
  }
  return launch_event_noalloc(g, n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin, status, st);
}

extern "C" int sim_run_batch_dev(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                                 const uint16_t *place, int64_t ld_place, const int32_t *gap,
                                 const int32_t *delay, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                                 int32_t *status, uint32_t flags, void *stream) {
  if (!g || n_scen < 0 || (flags != SIM_ALGO_AUTO && flags != SIM_ALGO_EVENT)) return SIM_E_INVAL;
  for (int32_t r = 0; r < g->n_res; ++r)
    if ((gap && gap[r] < 0) || (delay && delay[r] < 0)) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (bad_matrix(dur, ld_dur, n_scen, g->n_ops)) return SIM_E_INVAL;
  if (place && ld_place < n_scen) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  if (g->n_ops == 0) {
    if (launch_zero(makespan, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    if (status && launch_zero(status, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    return SIM_OK;
  }
  Lease lease(g->pool, st);
  if (lease.rc()) return lease.rc();
  if (!gap && !delay)
    return launch_event(g, lease.base(), n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin,
                        status, st);
  // gaps then delays go to the call's scratch set in stream order before the
  // replay, passed by value, so the caller's arrays are no longer read on
  // return
  const int32_t R = g->n_res;
  std::vector<int32_t> words((size_t)2 * R, 0);
  for (int32_t r = 0; r < R; ++r) {
    if (gap) words[r] = gap[r];
    if (delay) words[R + r] = delay[r];
  }
  int32_t *dev = (int32_t *)(lease.base() + g->scratch_dev_off);
  if (int rc = launch_put_words(dev, words.data(), 2 * R, st)) return rc;
  return launch_event_dev(g, lease.base(), n_scen, dur, ld_dur, place, ld_place, dev, gap != nullptr,
                          delay != nullptr, makespan, finish, ld_fin, status, st);
}

extern "C" int sim_run_batch_share(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                                   const uint8_t *share, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                                   int32_t *status, void *stream) {
  if (!g || n_scen < 0) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (bad_matrix(dur, ld_dur, n_scen, g->n_ops)) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  if (g->n_ops == 0) {
    if (launch_zero(makespan, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    if (status && launch_zero(status, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    return SIM_OK;
  }
  bool any = false;
  std::vector<int32_t> words((size_t)g->n_res, 0);
  for (int32_t r = 0; r < g->n_res; ++r) {
    words[r] = share && share[r] ? 1 : 0;
    any = any || words[r];
  }
  if (!any) {  // nothing shared: the plain replay
    Lease lease(g->pool, st);
    if (lease.rc()) return lease.rc();
    return launch_event(g, lease.base(), n_scen, dur, ld_dur, nullptr, 0, makespan, finish, ld_fin, status,
                        st);
  }
  Lease lease(g->share_pool, st);
  if (lease.rc()) return lease.rc();
  return launch_share(g, lease.base(), n_scen, dur, ld_dur, words.data(), makespan, finish, ld_fin, status,
                      st);
}

extern "C" int sim_run_batch_gap(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                                 const uint16_t *place, int64_t ld_place, const int32_t *gap,
                                 int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                                 uint32_t flags, void *stream) {
  if (!gap) return SIM_E_INVAL;
  return sim_run_batch_dev(g, n_scen, dur, ld_dur, place, ld_place, gap, nullptr, makespan, finish, ld_fin,
                           status, flags, stream);
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
    if (launch_zero(cp_len, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    if (path_scen >= 0) *path_len = 0;
    return SIM_OK;
  }
  // the path's dist column stays in the call's set until the copy below
  Lease lease(g->pool, st);
  if (lease.rc()) return lease.rc();
  int32_t *dist_dev = path_scen >= 0 ? (int32_t *)(lease.base() + g->scratch_dist_off) : nullptr;
  int rc = launch_cp(g, lease.base(), n_scen, dur, ld_dur, cp_len, dist_dev, path_scen, st);
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
  walk_critical_path(g, dist, d, cp_s, path_ops, path_cap, path_len);
  return SIM_OK;
}

extern "C" int sim_generate(int32_t n_ops, int64_t n_scen, const int32_t *base, int32_t n_knobs,
                            int64_t knob_block, uint32_t noise, uint64_t seed, int64_t scen0,
                            int32_t *dur, int64_t ld_dur, void *stream) {
  if (n_ops < 0 || n_scen < 0) return SIM_E_INVAL;
  DurGen gen;
  if (int rc = make_gen(n_ops, n_scen, base, n_knobs, knob_block, noise, seed, scen0, gen)) return rc;
  if (n_ops == 0 || n_scen == 0) return SIM_OK;
  if (bad_matrix(dur, ld_dur, n_scen, n_ops)) return SIM_E_INVAL;
  return launch_generate(gen, n_scen, dur, ld_dur, (hipStream_t)stream);
}

extern "C" int sim_run_generated(const sim_graph *g, int64_t n_scen, const int32_t *base, int32_t n_knobs,
                                 int64_t knob_block, uint32_t noise, uint64_t seed, int64_t scen0,
                                 int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                                 uint32_t flags, void *stream) {
  if (!g || n_scen < 0 || (flags != SIM_ALGO_AUTO && flags != SIM_ALGO_EVENT)) return SIM_E_INVAL;
  DurGen gen;
  if (int rc = make_gen(g->n_ops, n_scen, base, n_knobs, knob_block, noise, seed, scen0, gen)) return rc;
  if (n_scen == 0) return SIM_OK;
  if (!makespan) return SIM_E_INVAL;
  if (finish && ld_fin < n_scen) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  if (g->n_ops == 0) {
    if (launch_zero(makespan, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    if (status && launch_zero(status, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    return SIM_OK;
  }
  Lease lease(g->pool, st);
  if (lease.rc()) return lease.rc();
  return launch_event_gen(g, lease.base(), n_scen, gen, makespan, finish, ld_fin, status, st);
}

extern "C" int sim_critical_path_generated(const sim_graph *g, int64_t n_scen, const int32_t *base,
                                           int32_t n_knobs, int64_t knob_block, uint32_t noise,
                                           uint64_t seed, int64_t scen0, int32_t *cp_len,
                                           int64_t path_scen, int32_t *path_ops, int32_t path_cap,
                                           int32_t *path_len, void *stream) {
  if (!g || n_scen < 0) return SIM_E_INVAL;
  if (path_scen >= n_scen || path_scen < -1) return SIM_E_INVAL;
  if (path_scen >= 0 && (!path_len || (path_cap > 0 && !path_ops) || path_cap < 0)) return SIM_E_INVAL;
  DurGen gen;
  if (int rc = make_gen(g->n_ops, n_scen, base, n_knobs, knob_block, noise, seed, scen0, gen)) return rc;
  if (n_scen == 0) return SIM_OK;
  if (!cp_len) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  const int32_t n = g->n_ops;
  if (n == 0) {
    if (launch_zero(cp_len, n_scen, n_scen, 1, st) != SIM_OK) return SIM_E_HIP;
    if (path_scen >= 0) *path_len = 0;
    return SIM_OK;
  }
  Lease lease(g->pool, st);
  if (lease.rc()) return lease.rc();
  int32_t *dist_dev = path_scen >= 0 ? (int32_t *)(lease.base() + g->scratch_dist_off) : nullptr;
  int rc = launch_cp(g, lease.base(), n_scen, nullptr, 0, cp_len, dist_dev, path_scen, st, &gen);
  if (rc || path_scen < 0) return rc;
  // the path scenario's durations, generated once more into the call's set
  int32_t *dcol = (int32_t *)(lease.base() + g->scratch_gen_off);
  DurGen one = gen;
  one.scen0 = gen.scen0 + path_scen;
  if ((rc = launch_generate(one, 1, dcol, 1, st))) return rc;
  std::vector<int32_t> dist(n), d(n);
  int32_t cp_s = 0;
  if (hipMemcpyAsync(dist.data(), dist_dev, (size_t)n * 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(d.data(), dcol, (size_t)n * 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(&cp_s, cp_len + path_scen, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return SIM_E_HIP;
  walk_critical_path(g, dist, d, cp_s, path_ops, path_cap, path_len);
  return SIM_OK;
}

extern "C" int sim_attribute(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                             const uint16_t *place, int64_t ld_place, int32_t *makespan,
                             int32_t *status, int32_t *finish, int32_t *prev, int64_t ld_op,
                             int32_t *busy, int32_t *chain, int64_t ld_res, int32_t *chain_ops,
                             int64_t path_scen, int32_t *path_ops, int32_t path_cap,
                             int32_t *path_len, void *stream) {
  if (!g || n_scen < 0) return SIM_E_INVAL;
  if (path_scen >= n_scen || path_scen < -1) return SIM_E_INVAL;
  if (path_scen >= 0 && (!path_len || (path_cap > 0 && !path_ops) || path_cap < 0)) return SIM_E_INVAL;
  if (n_scen == 0) return SIM_OK;
  if (!makespan || !status || !chain_ops || !busy || !chain || ld_res < n_scen) return SIM_E_INVAL;
  const int32_t n = g->n_ops, R = g->n_res;
  if (n > 0 && (!finish || !prev || ld_op < n_scen)) return SIM_E_INVAL;
  if (bad_matrix(dur, ld_dur, n_scen, n)) return SIM_E_INVAL;
  if (place && ld_place < n_scen) return SIM_E_INVAL;
  hipStream_t st = (hipStream_t)stream;
  if (n == 0) {
    // no ops: every iteration takes 0 ns on an empty chain
    if (launch_zero(makespan, n_scen, n_scen, 1, st) != SIM_OK ||
        launch_zero(status, n_scen, n_scen, 1, st) != SIM_OK ||
        launch_zero(chain_ops, n_scen, n_scen, 1, st) != SIM_OK ||
        launch_zero(busy, n_scen, ld_res, R, st) != SIM_OK || launch_zero(chain, n_scen, ld_res, R, st) != SIM_OK)
      return SIM_E_HIP;
    if (path_scen >= 0) *path_len = 0;
    return SIM_OK;
  }
  int rc;
  {
    Lease lease(g->pool, st);
    if (lease.rc()) return lease.rc();
    rc = launch_event_prev(g, lease.base(), n_scen, dur, ld_dur, place, ld_place, makespan, finish, prev,
                           ld_op, status, st);
    if (rc) return rc;
    rc = launch_attr(g, lease.base(), n_scen, dur, ld_dur, place, ld_place, finish, prev, ld_op, status, busy,
                     chain, ld_res, chain_ops, st);
  }
  if (rc || path_scen < 0) return rc;

  // the chain of one scenario, walked on the host by the kernel's rule
  std::vector<int32_t> f(n), d(n), pv(n), res(n);
  std::vector<uint16_t> pl(place ? n : 0);
  int32_t st_s = 0;
  const int64_t ps = path_scen;
  if (hipMemcpy2DAsync(f.data(), 4, finish + ps, (size_t)ld_op * 4, 4, n, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpy2DAsync(d.data(), 4, dur + ps, (size_t)ld_dur * 4, 4, n, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpy2DAsync(pv.data(), 4, prev + ps, (size_t)ld_op * 4, 4, n, hipMemcpyDeviceToHost, st) != hipSuccess ||
      (place && hipMemcpy2DAsync(pl.data(), 2, place + ps, (size_t)ld_place * 2, 2, n, hipMemcpyDeviceToHost,
                                 st) != hipSuccess) ||
      hipMemcpyAsync(&st_s, status + ps, 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return SIM_E_HIP;
  *path_len = 0;
  if (st_s) return SIM_OK;
  // predecessors by caller id
  std::vector<std::vector<int32_t>> pred(n);
  for (int32_t c = 0; c < n; ++c)
    for (int32_t k = g->h_pred_ptr[c]; k < g->h_pred_ptr[c + 1]; ++k)
      pred[g->h_orig_of[c]].push_back(g->h_orig_of[g->h_pred[k]]);
  int32_t v = 0;
  for (int32_t x = 1; x < n; ++x)
    if (f[x] > f[v]) v = x;
  std::vector<int32_t> rev;
  while (v >= 0 && v < n && (int32_t)rev.size() < n) {
    rev.push_back(v);
    const int32_t start = f[v] - d[v];
    if (start <= 0) break;
    int32_t nxt = -1;
    for (int32_t p : pred[v])
      if (f[p] == start && (nxt < 0 || p < nxt)) nxt = p;
    v = nxt >= 0 ? nxt : pv[v];
  }
  *path_len = (int32_t)rev.size();
  for (int32_t k = 0; k < (int32_t)rev.size() && k < path_cap; ++k) path_ops[k] = rev[rev.size() - 1 - k];
  return SIM_OK;
}
