// Graph compilation (host): validation, duplicate-edge removal, cycle check,
// transitive reduction, renumbering by (priority, id), bounds used to size
// per-lane state, the critical-path sweep order with its value slots, and the
// upload of everything to one device allocation.
//
// The paper's preprocessing module turns framework graphs into one unified
// format before simulation (Sec. 2, "Overall System"); successor CSR with an
// op -> resource map is that format here.
#include <algorithm>
#include <cstring>
#include <iterator>
#include <map>
#include <new>
#include <numeric>
#include <queue>
#include <vector>

#include "sim.hpp"
#include "mlsim_testing.h"

using namespace mlsim;

namespace {

constexpr int32_t kReduceMaxOps = 32768;  // transitive reduction bitsets: n^2/8 bytes

struct Compiled {
  std::vector<OpRec> ops;
  std::vector<int32_t> succ, jneed, src, cp_pred, pred_ptr, pred, topo;
  std::vector<int32_t> lvl_of, levend;  // sweep variant: level of each op, last position of each level
  std::vector<int32_t> jtarget;  // [J] the op a join releases: its own op, or a barrier's first member
  // event kernel: records and successor entries holding heap-key words,
  // {predecessors needed, word released} per join, source words
  std::vector<OpRec> ev_ops;
  std::vector<int32_t> ev_succ, jinfo, ev_src;
  int32_t pk_sh = 0, pk_join = 0, pk_jn = 0, pk_jb = 0, pk_rb = 0, ev_compact = 0, pk_rkey = 0;
  std::vector<int32_t> ev_rec16;  // [n][4] compact event records (ev_compact)
  std::vector<int32_t> wp_ptr, wp, ws_ptr, ws;  // walk: predecessors / successors, barriers as nodes
  std::vector<CpRec> cp;
  std::vector<int32_t> jslot;    // [J] join state slot of each join (the event kernel's join index)
  std::vector<int32_t> join_of;  // [n] the join a compact op waits on (its own or its barrier's), -1
  int32_t J = 0, JS = 0, heap_cap = 0, cp_slots = 0, cp_n = 0, max_indeg = 0, levels = 0, barriers = 0;
  int64_t m = 0;
};

// Hopcroft-Karp maximum matching between "u has a successor" and "v has a
// predecessor" on the edges u -> v.  n - matching = minimum number of
// vertex-disjoint paths covering the DAG, an upper bound on any antichain
// (each path meets an antichain at most once), hence on how many ops can be
// ready at the same time.
int32_t min_path_cover(int32_t n, const std::vector<std::vector<int32_t>> &adj) {
  std::vector<int32_t> mu(n, -1), mv(n, -1), dist(n), it(n), q(n);
  const int32_t INF = INT32_MAX;
  int32_t matched = 0;
  for (;;) {
    int32_t qh = 0, qt = 0;
    bool found = false;
    for (int32_t u = 0; u < n; ++u) {
      if (mu[u] < 0) {
        dist[u] = 0;
        q[qt++] = u;
      } else {
        dist[u] = INF;
      }
    }
    while (qh < qt) {
      int32_t u = q[qh++];
      for (int32_t v : adj[u]) {
        int32_t w = mv[v];
        if (w < 0) {
          found = true;
        } else if (dist[w] == INF) {
          dist[w] = dist[u] + 1;
          q[qt++] = w;
        }
      }
    }
    if (!found) break;
    // iterative DFS along layered augmenting paths
    std::vector<int32_t> stack;
    for (int32_t u = 0; u < n; ++u) it[u] = 0;
    for (int32_t root = 0; root < n; ++root) {
      if (mu[root] >= 0) continue;
      stack.assign(1, root);
      while (!stack.empty()) {
        int32_t u = stack.back();
        if (it[u] >= (int32_t)adj[u].size()) {
          dist[u] = INF;
          stack.pop_back();
          continue;
        }
        int32_t v = adj[u][it[u]];
        int32_t w = mv[v];
        if (w < 0) {
          // augment along the stack
          for (int32_t k = (int32_t)stack.size() - 1; k >= 0; --k) {
            int32_t uu = stack[k];
            int32_t vv = adj[uu][it[uu]];
            int32_t prev = mu[uu];
            mu[uu] = vv;
            mv[vv] = uu;
            (void)prev;
          }
          ++matched;
          stack.clear();
        } else if (dist[w] == dist[u] + 1) {
          stack.push_back(w);
        } else {
          ++it[u];
        }
      }
    }
  }
  return n - matched;
}

// Join state slots of the event replay.  A join's state {predecessors
// finished, latest finish} is live from the completion of its first
// predecessor until that of its last one, which clears it.  Join k may take
// over the slot of join j when j's node is an ancestor-or-self of every
// predecessor of k: each predecessor of k then completes after j's node was
// released, hence after j's last predecessor cleared j's state, so the two
// are never open together, whatever the durations.  (Siblings of one op
// never qualify: neither is an ancestor of their common predecessor.)  Joins
// are visited in a topological order of the walk graph (nodes 0..N-1, preds
// / succs as CSR) and take the lowest slot whose latest holder qualifies,
// else a new one.  Ancestor sets (bitsets over join ids) are kept only while
// a successor of their node is unvisited; when they would need more than
// kJoinSlotBudget bytes, every join keeps a slot of its own.  Only the
// first kJoinSlotScan slots are tried for each join (a bound on the time).
constexpr size_t kJoinSlotBudget = size_t(256) << 20;
constexpr size_t kJoinSlotScan = 4096;

int32_t assign_join_slots(int32_t N, const std::vector<int32_t> &p_ptr, const std::vector<int32_t> &p,
                          const std::vector<int32_t> &s_ptr, const std::vector<int32_t> &s,
                          const std::vector<int32_t> &jid, int32_t J, std::vector<int32_t> &slot) {
  slot.resize(J);
  std::iota(slot.begin(), slot.end(), 0);
  if (J <= 1) return J;
  const size_t W = ((size_t)J + 63) / 64;
  std::vector<int32_t> cnt(N), left(N), order;
  order.reserve(N);
  for (int32_t x = 0; x < N; ++x) {
    cnt[x] = p_ptr[x + 1] - p_ptr[x];
    left[x] = s_ptr[x + 1] - s_ptr[x];
    if (cnt[x] == 0) order.push_back(x);
  }
  std::vector<std::vector<uint64_t>> anc(N);
  std::vector<int32_t> holder;  // per slot: its latest join
  std::vector<uint64_t> ca(W);
  size_t live = 0;
  for (size_t h = 0; h < order.size(); ++h) {
    const int32_t x = order[h];
    std::vector<uint64_t> a(W, 0);
    std::fill(ca.begin(), ca.end(), ~0ull);
    for (int32_t e = p_ptr[x]; e < p_ptr[x + 1]; ++e) {
      const std::vector<uint64_t> &b = anc[p[e]];
      for (size_t w = 0; w < W; ++w) {
        a[w] |= b[w];
        ca[w] &= b[w];
      }
    }
    for (int32_t e = p_ptr[x]; e < p_ptr[x + 1]; ++e)
      if (--left[p[e]] == 0) {
        std::vector<uint64_t>().swap(anc[p[e]]);
        live -= W * 8;
      }
    const int32_t j = jid[x];
    if (j >= 0) {
      const size_t scan = std::min(holder.size(), kJoinSlotScan);
      size_t k = 0;
      while (k < scan && !(ca[(size_t)holder[k] / 64] >> (holder[k] % 64) & 1)) ++k;
      if (k == scan) k = holder.size();
      if (k == holder.size()) holder.push_back(j);
      holder[k] = j;
      slot[j] = (int32_t)k;
      a[(size_t)j / 64] |= 1ull << (j % 64);
    }
    if (left[x] > 0) {
      anc[x].swap(a);
      live += W * 8;
      if (live > kJoinSlotBudget) {
        std::iota(slot.begin(), slot.end(), 0);
        return J;
      }
    }
    for (int32_t e = s_ptr[x]; e < s_ptr[x + 1]; ++e)
      if (--cnt[s[e]] == 0) order.push_back(s[e]);
  }
  return (int32_t)holder.size();
}

// Kahn's algorithm; lifo = depth-first flavour.  Returns false on a cycle.
bool kahn(int32_t n, const std::vector<std::vector<int32_t>> &succ, bool lifo,
          std::vector<int32_t> &order) {
  std::vector<int32_t> cnt(n, 0);
  for (int32_t u = 0; u < n; ++u)
    for (int32_t w : succ[u]) cnt[w]++;
  std::vector<int32_t> work;
  order.clear();
  order.reserve(n);
  size_t head = 0;
  for (int32_t v = n - 1; v >= 0; --v)
    if (cnt[v] == 0) work.push_back(v);
  if (!lifo) std::reverse(work.begin(), work.end());
  while (lifo ? !work.empty() : head < work.size()) {
    int32_t v;
    if (lifo) {
      v = work.back();
      work.pop_back();
    } else {
      v = work[head++];
    }
    order.push_back(v);
    const auto &s = succ[v];
    for (int32_t k = (int32_t)s.size() - 1; k >= 0; --k)
      if (--cnt[s[k]] == 0) work.push_back(s[k]);
  }
  return (int32_t)order.size() == n;
}

// Slots for the critical-path sweep in `order`: dist(v) lives from v's
// position to its last successor's position.
int32_t assign_cp_slots(int32_t n, const std::vector<std::vector<int32_t>> &succ,
                        const std::vector<std::vector<int32_t>> &pred,
                        const std::vector<int32_t> &order, std::vector<int32_t> &slot_of) {
  std::vector<int32_t> pos(n), last(n, -1);
  for (int32_t k = 0; k < n; ++k) pos[order[k]] = k;
  for (int32_t v = 0; v < n; ++v)
    for (int32_t w : succ[v]) last[v] = std::max(last[v], pos[w]);
  slot_of.assign(n, -1);
  std::vector<int32_t> freel;
  int32_t nslots = 0;
  for (int32_t k = 0; k < n; ++k) {
    int32_t v = order[k];
    for (int32_t p : pred[v])
      if (last[p] == k) freel.push_back(slot_of[p]);
    if (!succ[v].empty()) {
      if (freel.empty()) {
        slot_of[v] = nslots++;
      } else {
        slot_of[v] = freel.back();
        freel.pop_back();
      }
    }
  }
  return nslots;
}

// A topological order that keeps few values live: among the ready nodes,
// visit the one that ends the most live values (predecessors whose last
// unvisited successor it is), less one if its own value will be live;
// ties go to the smaller tie key.  Scores only grow while a node waits
// (a predecessor reaching its last unvisited successor adds one to that
// successor), so each change pushes a fresh heap entry and stale entries are
// skipped: O((nodes + edges) log nodes).
void greedy_order(int32_t n, const std::vector<std::vector<int32_t>> &succ,
                  const std::vector<std::vector<int32_t>> &pred, const std::vector<int64_t> &tie,
                  std::vector<int32_t> &order) {
  std::vector<int32_t> cnt(n), rem(n), score(n);
  std::vector<char> done(n, 0);
  for (int32_t v = 0; v < n; ++v) {
    cnt[v] = (int32_t)pred[v].size();
    rem[v] = (int32_t)succ[v].size();
    score[v] = succ[v].empty() ? 0 : -1;
  }
  for (int32_t v = 0; v < n; ++v)
    for (int32_t p : pred[v])
      if (rem[p] == 1) ++score[v];
  struct Entry {
    int32_t score;
    int64_t tie;
    int32_t v;
    bool operator<(const Entry &o) const {  // max-heap: higher score, then smaller tie
      return score != o.score ? score < o.score : tie > o.tie;
    }
  };
  std::priority_queue<Entry> heap;
  for (int32_t v = 0; v < n; ++v)
    if (cnt[v] == 0) heap.push({score[v], tie[v], v});
  order.clear();
  order.reserve(n);
  while (!heap.empty()) {
    const Entry e = heap.top();
    heap.pop();
    if (done[e.v] || e.score != score[e.v]) continue;
    const int32_t v = e.v;
    done[v] = 1;
    order.push_back(v);
    for (int32_t p : pred[v])
      if (--rem[p] == 1)
        for (int32_t q : succ[p])
          if (!done[q]) {
            ++score[q];
            if (cnt[q] == 0) heap.push({score[q], tie[q], q});
            break;
          }
    for (int32_t w : succ[v])
      if (--cnt[w] == 0) heap.push({score[w], tie[w], w});
  }
}

int compile(int32_t n, int32_t R, const int64_t *succ_ptr, const int32_t *succ_idx,
            const int32_t *op_res, const int32_t *prio, Compiled &C) {
  // deduplicated successor lists
  std::vector<std::vector<int32_t>> succ(n);
  for (int32_t u = 0; u < n; ++u) {
    succ[u].assign(succ_idx + succ_ptr[u], succ_idx + succ_ptr[u + 1]);
    std::sort(succ[u].begin(), succ[u].end());
    succ[u].erase(std::unique(succ[u].begin(), succ[u].end()), succ[u].end());
  }
  std::vector<int32_t> topo;
  if (!kahn(n, succ, false, topo)) return SIM_E_CYCLE;
  std::vector<int32_t> pos(n);
  for (int32_t k = 0; k < n; ++k) pos[topo[k]] = k;

  // Transitive reduction: drop u -> w when w is reachable from another
  // successor of u.  The later of the two predecessors on that path always
  // finishes after u (durations >= 1), so every ready time is unchanged, and
  // every op still becomes ready when its last remaining predecessor ends.
  if (n <= kReduceMaxOps) {
    const size_t words = ((size_t)n + 63) / 64;
    std::vector<uint64_t> reach;
    try {
      reach.assign(words * (size_t)n, 0);
    } catch (const std::bad_alloc &) {
      return SIM_E_NOMEM;
    }
    std::vector<uint64_t> acc(words);
    for (int32_t k = n - 1; k >= 0; --k) {
      int32_t u = topo[k];
      auto &s = succ[u];
      std::sort(s.begin(), s.end(), [&](int32_t a, int32_t b) { return pos[a] < pos[b]; });
      std::fill(acc.begin(), acc.end(), 0);
      std::vector<int32_t> keep;
      for (int32_t w : s) {
        size_t bit = (size_t)pos[w];
        if ((acc[bit >> 6] >> (bit & 63)) & 1) continue;
        keep.push_back(w);
        const uint64_t *rw = &reach[(size_t)w * words];
        for (size_t i = 0; i < words; ++i) acc[i] |= rw[i];
        acc[bit >> 6] |= 1ull << (bit & 63);
      }
      std::copy(acc.begin(), acc.end(), reach.begin() + (size_t)u * words);
      s.swap(keep);
    }
  }

  // renumber by (priority, id): compact id order is the tie-break order
  std::vector<int32_t> orig_of(n), comp(n);
  std::iota(orig_of.begin(), orig_of.end(), 0);
  if (prio)
    std::stable_sort(orig_of.begin(), orig_of.end(),
                     [&](int32_t a, int32_t b) { return prio[a] < prio[b]; });
  for (int32_t c = 0; c < n; ++c) comp[orig_of[c]] = c;

  std::vector<std::vector<int32_t>> cs(n), cp(n);  // compact successors / predecessors
  for (int32_t u = 0; u < n; ++u)
    for (int32_t w : succ[u]) {
      cs[comp[u]].push_back(comp[w]);
      cp[comp[w]].push_back(comp[u]);
    }
  for (int32_t c = 0; c < n; ++c) {
    std::sort(cs[c].begin(), cs[c].end());
    std::sort(cp[c].begin(), cp[c].end());
  }
  std::vector<int32_t> ctopo(n);
  for (int32_t k = 0; k < n; ++k) ctopo[k] = comp[topo[k]];

  // Successor structure of the event replay.  Ops sharing one predecessor
  // set of two or more ops wait on one barrier node (id n + b) instead of
  // each counting the same predecessors: a barrier completes when its last
  // predecessor finishes and releases its members at that instant, so every
  // ready time is unchanged.
  std::vector<std::vector<int32_t>> es(cs);  // successors, barriers included
  std::vector<int32_t> need(n);
  for (int32_t c = 0; c < n; ++c) need[c] = (int32_t)cp[c].size();
  std::map<std::vector<int32_t>, std::vector<int32_t>> groups;
  for (int32_t c = 0; c < n; ++c)
    if (cp[c].size() >= 2) groups[cp[c]].push_back(c);
  std::vector<std::vector<int32_t>> bmem;
  std::vector<int32_t> bneed;
  for (auto &kv : groups) {
    if (kv.second.size() < 2) continue;
    const int32_t b = n + (int32_t)bmem.size();
    for (int32_t p : kv.first) {
      std::vector<int32_t> keep;
      std::set_difference(es[p].begin(), es[p].end(), kv.second.begin(), kv.second.end(),
                          std::back_inserter(keep));
      keep.push_back(b);  // ids above n keep the list sorted
      es[p].swap(keep);
    }
    for (int32_t w : kv.second) need[w] = 1;
    bmem.push_back(kv.second);
    bneed.push_back((int32_t)kv.first.size());
  }
  const int32_t nb = (int32_t)bmem.size();
  C.barriers = nb;
  // A barrier's members share one ready time, so they leave the ready list in
  // compact-id order one after another.  The barrier releases only its first
  // member; popping member i releases member i + 1 at the same ready time
  // (a "sibling" entry, first in its list).  The ready list then holds one
  // entry per completed barrier instead of all its members, and the pop
  // order is unchanged: the held-back members are never the minimum.
  for (int32_t b = 0; b < nb; ++b) {
    const auto &mem = bmem[b];
    for (size_t i = 0; i + 1 < mem.size(); ++i) es[mem[i]].insert(es[mem[i]].begin(), mem[i + 1]);
  }
  // Fans: the successors of an op p whose only predecessor is p share p's
  // output time as their ready time, so they too can be chained: p releases
  // the first, and popping member i releases member i + 1 (the pop order is
  // unchanged by the argument above; members are chained in compact-id
  // order, which is their key order).  Chained only where p has more than
  // two entries (two are held in its record, the rest read one after
  // another from the successor list) and only members whose own list is at
  // most one entry, so each member still holds its entries in its record.
  // (A member's join then follows its sibling entry, so its state is read
  // after the record instead of with it: one round trip in the member's
  // step against the list reads saved in p's.)
  std::vector<std::vector<int32_t>> fans;
  for (int32_t p = 0; p < n; ++p) {
    if (es[p].size() <= 2) continue;
    std::vector<int32_t> mem;
    for (int32_t w : es[p])
      if (w < n && need[w] == 1 && cp[w].size() == 1 && es[w].size() <= 1)
        mem.push_back(w);
    if (mem.size() < 2) continue;
    std::sort(mem.begin(), mem.end());
    // (order kept: p may be a barrier member whose sibling entry comes first)
    std::vector<int32_t> keep;
    for (int32_t x : es[p])
      if (x == mem[0] || !std::binary_search(mem.begin() + 1, mem.end(), x)) keep.push_back(x);
    es[p].swap(keep);
    for (size_t i = 0; i + 1 < mem.size(); ++i) es[mem[i]].insert(es[mem[i]].begin(), mem[i + 1]);
    fans.push_back(std::move(mem));
  }

  // Walk graph (pull model): node ids are the compact ops 0..n-1 and the
  // barriers n..n+nb-1.  A barrier's predecessors are its shared set; each
  // member has the barrier as its only predecessor; every other op keeps its
  // reduced predecessors.  Successor lists are the reverse.
  {
    const int32_t N = n + nb;
    std::vector<int32_t> bar_of(n, -1);
    for (int32_t b = 0; b < nb; ++b)
      for (int32_t w : bmem[b]) bar_of[w] = n + b;
    std::vector<std::vector<int32_t>> wpl(N);
    for (int32_t c = 0; c < n; ++c) {
      if (bar_of[c] >= 0)
        wpl[c].push_back(bar_of[c]);
      else
        wpl[c] = cp[c];
    }
    for (auto &kv : groups)
      if (kv.second.size() >= 2) wpl[bar_of[kv.second[0]]] = kv.first;
    std::vector<std::vector<int32_t>> wsl(N);
    for (int32_t x = 0; x < N; ++x)
      for (int32_t p : wpl[x]) wsl[p].push_back(x);
    C.wp_ptr.assign(N + 1, 0);
    C.ws_ptr.assign(N + 1, 0);
    C.wp.clear();
    C.ws.clear();
    for (int32_t x = 0; x < N; ++x) {
      C.wp_ptr[x] = (int32_t)C.wp.size();
      C.wp.insert(C.wp.end(), wpl[x].begin(), wpl[x].end());
      C.ws_ptr[x] = (int32_t)C.ws.size();
      C.ws.insert(C.ws.end(), wsl[x].begin(), wsl[x].end());
    }
    C.wp_ptr[N] = (int32_t)C.wp.size();
    C.ws_ptr[N] = (int32_t)C.ws.size();
  }

  // joins: ops still counting two or more predecessors, in topological
  // order, then the barriers; their state slots may be shared (see
  // assign_join_slots)
  std::vector<int32_t> join(n + nb, -1);  // kJoinNone for plain successors
  C.J = 0;
  C.jneed.clear();
  C.jtarget.clear();
  for (int32_t k = 0; k < n; ++k)
    if (need[ctopo[k]] >= 2) {
      join[ctopo[k]] = C.J++;
      C.jneed.push_back(need[ctopo[k]]);
      C.jtarget.push_back(ctopo[k]);
    }
  for (int32_t b = 0; b < nb; ++b) {
    join[n + b] = C.J++;
    C.jneed.push_back(bneed[b]);
    C.jtarget.push_back(bmem[b][0]);
  }
  C.join_of.assign(join.begin(), join.begin() + n);
  for (int32_t b = 0; b < nb; ++b)
    for (int32_t w : bmem[b]) C.join_of[w] = join[n + b];
  C.JS = assign_join_slots(n + nb, C.wp_ptr, C.wp, C.ws_ptr, C.ws, join, C.J, C.jslot);
  C.max_indeg = 0;
  for (int32_t c = 0; c < n; ++c) C.max_indeg = std::max(C.max_indeg, (int32_t)cp[c].size());

  // records and successor entries {id, join index or -1}
  C.ops.resize(n + nb + 1);
  C.succ.clear();
  int32_t e = 0;
  // sibling entries: the first entry of a barrier or fan member that has a next one
  std::vector<uint8_t> has_sib(n, 0);
  for (int32_t b = 0; b < nb; ++b)
    for (size_t i = 0; i + 1 < bmem[b].size(); ++i) has_sib[bmem[b][i]] = 1;
  for (const auto &mem : fans)
    for (size_t i = 0; i + 1 < mem.size(); ++i) has_sib[mem[i]] = 1;
  for (int32_t c = 0; c < n + nb; ++c) {
    std::vector<int32_t> lst = c < n ? es[c] : std::vector<int32_t>{bmem[c - n][0]};
    std::vector<int32_t> jl(lst.size());
    for (size_t k = 0; k < lst.size(); ++k) jl[k] = join[lst[k]];
    if (c < n && has_sib[c]) jl[0] = kJoinSibling;
    OpRec r{c < n ? orig_of[c] : -1, c < n ? op_res[orig_of[c]] : -1, e, (int32_t)lst.size(),
            -1, -1, 0, 0};
    if (!lst.empty()) {
      r.w0 = lst[0];
      r.j0 = jl[0];
    }
    if (lst.size() > 1) {
      r.w1 = lst[1];
      r.j1 = jl[1];
    }
    C.ops[c] = r;
    for (size_t k = 0; k < lst.size(); ++k) {
      C.succ.push_back(lst[k]);
      C.succ.push_back(jl[k]);
      ++e;
    }
  }
  C.ops[n + nb] = OpRec{-1, -1, e, 0, -1, -1, 0, 0};
  C.m = 0;
  for (int32_t c = 0; c < n; ++c) C.m += (int64_t)cs[c].size();
  C.src.clear();
  for (int32_t c = 0; c < n; ++c)
    if (cp[c].empty()) C.src.push_back(c);

  // Heap-key words of the event kernel.  The low 32 bits of a ready-list key
  // hold the compact id; when the bits allow, they also hold (below it) the
  // op's resource and the join index of its first successor entry (all
  // ones: not a join), so a popped op's first join state can be read
  // together with its record instead of after it, and its resource without
  // its record.  The id in the top bits keeps the key order (ids are
  // distinct).  (A second join field for the second entry did not measure
  // faster on the BERT workload.)
  {
    // A join entry can carry everything its firing needs: the word of the op
    // it releases and, beside the join index, the number of predecessors it
    // waits for (when they fit 16 and 15 bits), so no per-join table is read.
    // The join field of an entry and of a key word is the join's state slot;
    // without self-contained entries it also indexes the per-join table, so
    // every join then keeps a slot of its own.
    bool jn = C.JS <= 65536;
    for (int32_t j = 0; j < C.J && jn; ++j) jn = C.jneed[j] < 32768;
    if (!jn) {
      std::iota(C.jslot.begin(), C.jslot.end(), 0);
      C.JS = C.J;
    }
    C.pk_jn = jn;
    int32_t jb = 0, rb = 0;
    while ((1ll << jb) < (int64_t)C.JS + 1) ++jb;
    while ((1ll << rb) < (int64_t)R) ++rb;
    bool ident = true;  // caller ids equal compact ids: the duration row is the id
    for (int32_t c = 0; c < n && ident; ++c) ident = orig_of[c] == c;
    // compact records: identity rows, self-contained join entries, and id
    // and join field in one word; the resource too when it fits (rkey),
    // else the replay reads it by row (it needs none with a placement)
    const bool compact = ident && jn && jb < 32 && (int64_t)n <= (1ll << (32 - jb));
    const bool rkey = compact && rb + jb < 32 && (int64_t)n <= (1ll << (32 - rb - jb));
    const bool pack = compact || (jb > 0 && jb < 32 && (int64_t)n <= (1ll << (32 - jb)));
    if (!rkey) rb = 0;
    if (!pack) jb = 0;
    C.ev_compact = compact;
    C.pk_rkey = rkey;
    C.pk_jb = jb;
    C.pk_rb = rb;
    C.pk_sh = rb + jb;
    C.pk_join = jb > 0;
    const uint32_t jnone = (1u << jb) - 1u;
    auto word = [&](int32_t c) -> int32_t {  // c: a compact op id (never a barrier)
      if (!pack || c < 0 || c >= n) return c;
      const OpRec &r = C.ops[c];
      const uint32_t jf = r.nsucc > 0 && r.j0 >= 0 ? (uint32_t)C.jslot[r.j0] : jnone;
      const uint32_t res = rkey ? (uint32_t)r.res << jb : 0u;
      return (int32_t)(((uint32_t)c << (rb + jb)) | res | jf);
    };
    auto entry = [&](int32_t &x, int32_t &y) {
      if (y < 0) {
        x = word(x);  // released directly (or a sibling)
      } else if (jn) {
        x = word(C.jtarget[y]);
        y = (int32_t)((uint32_t)C.jslot[y] | ((uint32_t)C.jneed[y] << 16));
      }
    };
    C.ev_ops = C.ops;
    for (OpRec &r : C.ev_ops) {
      if (r.nsucc > 0) entry(r.w0, r.j0);
      if (r.nsucc > 1) entry(r.w1, r.j1);
    }
    C.ev_succ = C.succ;
    for (size_t k = 0; k + 1 < C.ev_succ.size(); k += 2) entry(C.ev_succ[k], C.ev_succ[k + 1]);
    C.jinfo.resize(2 * (size_t)C.J);
    for (int32_t j = 0; j < C.J; ++j) {
      C.jinfo[2 * j] = C.jneed[j];
      C.jinfo[2 * j + 1] = word(C.jtarget[j]);
    }
    C.ev_src.clear();
    for (int32_t c : C.src) C.ev_src.push_back(word(c));
    // compact records {entry 0, entry 1} per op: an entry {x, y} as in the
    // successor list, {0, kRecNoSucc} when absent; an op with three or more
    // successors keeps entry 0 and {index of its entry 1 in the successor
    // list, kRecMore - (successors - 1)}
    C.ev_rec16.assign(compact ? 4 * (size_t)n : 0, 0);
    for (int32_t c = 0; compact && c < n; ++c) {
      const OpRec &r = C.ev_ops[c];
      int32_t *q = &C.ev_rec16[4 * (size_t)c];
      q[1] = q[3] = kRecNoSucc;
      if (r.nsucc > 0) q[0] = r.w0, q[1] = r.j0;
      if (r.nsucc == 2) q[2] = r.w1, q[3] = r.j1;
      if (r.nsucc > 2) q[2] = r.sbeg + 1, q[3] = kRecMore - (r.nsucc - 1);
    }
  }

  C.heap_cap = n ? std::max(1, min_path_cover(n, cs)) : 0;

  // critical-path sweep
  std::vector<int32_t> order;
  build_maxplus(n, cs, cp, {}, {}, orig_of, C.cp, C.cp_pred, C.cp_slots, order, C.cp_n);

  // compact predecessor CSR (for the sweep variant) and level count
  C.pred_ptr.assign(n + 1, 0);
  C.pred.clear();
  for (int32_t c = 0; c < n; ++c) {
    C.pred_ptr[c] = (int32_t)C.pred.size();
    C.pred.insert(C.pred.end(), cp[c].begin(), cp[c].end());
  }
  C.pred_ptr[n] = (int32_t)C.pred.size();
  std::vector<int32_t> lvl(n, 0);
  C.levels = 0;
  for (int32_t k = 0; k < n; ++k) {
    int32_t v = order[k];
    for (int32_t p : cp[v]) lvl[v] = std::max(lvl[v], lvl[p] + 1);
    C.levels = std::max(C.levels, lvl[v] + 1);
  }
  // sweep-variant order: by level (longest path from a source), then id, so
  // every level is a contiguous range of positions
  C.topo.resize(n);
  for (int32_t c = 0; c < n; ++c) C.topo[c] = c;
  std::stable_sort(C.topo.begin(), C.topo.end(), [&](int32_t a, int32_t b) { return lvl[a] < lvl[b]; });
  C.lvl_of = lvl;
  C.levend.assign(std::max(C.levels, 1), -1);
  for (int32_t k = 0; k < n; ++k) C.levend[lvl[C.topo[k]]] = k;
  return SIM_OK;
}

template <class T>
size_t bytes_of(const std::vector<T> &v) {
  return v.size() * sizeof(T);
}

}  // namespace

namespace mlsim {

bool build_maxplus(int32_t n, const std::vector<std::vector<int32_t>> &succ,
                   const std::vector<std::vector<int32_t>> &pred, const std::vector<int32_t> &extra,
                   const std::vector<int64_t> &tie, const std::vector<int32_t> &row_of,
                   std::vector<CpRec> &rec, std::vector<int32_t> &plist, int32_t &slots,
                   std::vector<int32_t> &order, int32_t &n_sweep) {
  // A second candidate table: one barrier node for each predecessor set (two
  // or more ops, not counting an op's extra predecessor) that two or more
  // ops share.  Its dist is the max over the set (duration 0), and each op
  // sharing the set takes the barrier (and its extra predecessor) instead:
  // the same dist for every op, and the set's values are dead once the
  // barrier has read them.
  auto extra_of = [&](int32_t v) { return extra.empty() ? -1 : extra[v]; };
  std::map<std::vector<int32_t>, std::vector<int32_t>> sets;
  for (int32_t v = 0; v < n; ++v) {
    std::vector<int32_t> key;
    for (int32_t p : pred[v])
      if (p != extra_of(v)) key.push_back(p);
    if (key.size() < 2) continue;
    std::sort(key.begin(), key.end());
    sets[key].push_back(v);
  }
  std::vector<std::vector<int32_t>> fpred(pred), fsucc;
  for (const auto &kv : sets) {
    if (kv.second.size() < 2) continue;
    const int32_t b = (int32_t)fpred.size();
    fpred.push_back(kv.first);
    for (int32_t v : kv.second) {
      fpred[v].assign(1, b);
      if (extra_of(v) >= 0) fpred[v].push_back(extra_of(v));
    }
  }
  const int32_t nf = (int32_t)fpred.size();
  fsucc.resize(nf);
  for (int32_t v = 0; v < nf; ++v)
    for (int32_t p : fpred[v]) fsucc[p].push_back(v);
  // the candidate (graph; depth-first, breadth-first or greedy order) that
  // needs the fewest live value slots; ties keep the earlier candidate
  struct Cand {
    int32_t nodes;
    const std::vector<std::vector<int32_t>> *succ, *pred;
    std::vector<int32_t> order, slot;
    int32_t live;
  };
  std::vector<int64_t> key(nf);  // greedy ties: the given key (else the id), barriers first
  for (int32_t v = 0; v < nf; ++v) key[v] = v >= n ? -1 : tie.empty() ? v : tie[v];
  std::vector<Cand> cand;
  for (int f = 0; f < (nf > n ? 2 : 1); ++f)
    for (int how = 0; how < 3; ++how) {
      Cand c{f ? nf : n, f ? &fsucc : &succ, f ? &fpred : &pred, {}, {}, 0};
      if (how < 2) {
        if (!kahn(c.nodes, *c.succ, how == 0, c.order)) return false;
      } else {
        greedy_order(c.nodes, *c.succ, *c.pred, key, c.order);
        if ((int32_t)c.order.size() != c.nodes) return false;
      }
      c.live = assign_cp_slots(c.nodes, *c.succ, *c.pred, c.order, c.slot);
      cand.push_back(std::move(c));
    }
  size_t pick = 0;
  for (size_t i = 1; i < cand.size(); ++i)
    if (cand[i].live < cand[pick].live) pick = i;
  const Cand &C = cand[pick];
  const auto &P = *C.pred;
  order.clear();
  for (int32_t v : C.order)
    if (v < n) order.push_back(v);  // still topological for the ops themselves
  n_sweep = C.nodes;
  // two more slots: one that always holds 0 (unused inline predecessors
  // read it) and one that ops without successors write (never read)
  slots = C.live + 2;
  const int32_t zslot = slots - 2, sink = slots - 1;
  const int32_t pad = (C.nodes + kCpBatch - 1) / kCpBatch * kCpBatch + kCpBatch * kCpAhead;
  rec.assign(pad, CpRec{n ? row_of[0] : 0, sink, 0, 0, {zslot, zslot, zslot, zslot}});
  plist.clear();
  for (int32_t k = 0; k < C.nodes; ++k) {
    const int32_t v = C.order[k];
    CpRec r{v < n ? row_of[v] : -1, C.slot[v] >= 0 ? C.slot[v] : sink, (int32_t)P[v].size(),
            (int32_t)plist.size(), {zslot, zslot, zslot, zslot}};
    if (P[v].size() <= 4)
      for (size_t e = 0; e < P[v].size(); ++e) r.p[e] = C.slot[P[v][e]];
    else
      for (int32_t p : P[v]) plist.push_back(C.slot[p]);
    rec[k] = r;
  }
  if (plist.empty()) plist.push_back(0);
  return true;
}

}  // namespace mlsim


namespace {

// The argument checks of sim_graph_create.
int check_graph_args(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr, const int32_t *succ_idx,
                     const int32_t *op_res) {
  if (n_ops < 0 || n_res < 1) return SIM_E_INVAL;
  if (n_ops > SIM_MAX_OPS || n_res > SIM_MAX_RES) return SIM_E_LIMIT;
  if (n_ops > 0 && (!succ_ptr || !op_res)) return SIM_E_INVAL;
  if (n_ops > 0) {
    if (succ_ptr[0] != 0) return SIM_E_INVAL;
    for (int32_t v = 0; v < n_ops; ++v)
      if (succ_ptr[v + 1] < succ_ptr[v]) return SIM_E_INVAL;
    if (succ_ptr[n_ops] >= INT32_MAX) return SIM_E_LIMIT;
    if (succ_ptr[n_ops] > 0 && !succ_idx) return SIM_E_INVAL;
    for (int64_t e = 0; e < succ_ptr[n_ops]; ++e)
      if (succ_idx[e] < 0 || succ_idx[e] >= n_ops) return SIM_E_RANGE;
    for (int32_t v = 0; v < n_ops; ++v)
      if (op_res[v] < 0 || op_res[v] >= n_res) return SIM_E_RANGE;
  }
  return SIM_OK;
}

}  // namespace

extern "C" int sim_graph_create(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                                const int32_t *succ_idx, const int32_t *op_res,
                                const int32_t *prio, sim_graph **out) {
  if (!out) return SIM_E_INVAL;
  *out = nullptr;
  if (int rc = check_graph_args(n_ops, n_res, succ_ptr, succ_idx, op_res)) return rc;
  Compiled C;
  int rc;
  try {
    rc = compile(n_ops, n_res, succ_ptr, succ_idx, op_res, prio, C);
  } catch (const std::bad_alloc &) {
    return SIM_E_NOMEM;
  }
  if (rc) return rc;
  if (C.max_indeg >= 65536) return SIM_E_LIMIT;

  sim_graph *g = new (std::nothrow) sim_graph();
  if (!g) return SIM_E_NOMEM;
  g->n_ops = n_ops;
  g->n_res = n_res;
  g->n_edges = C.m;
  g->n_joins = C.J;
  g->n_levels = C.levels;
  if (hipGetDevice(&g->device) != hipSuccess) {
    delete g;
    return SIM_E_HIP;
  }

  // one device allocation, 256-byte aligned pieces
  size_t off = 0;
  auto take = [&](size_t b) {
    size_t o = off;
    off += (b + 255) & ~size_t(255);
    return o;
  };
  size_t o_ops = take(bytes_of(C.ops)), o_succ = take(bytes_of(C.succ)),
         o_jneed = take(bytes_of(C.jneed)), o_src = take(bytes_of(C.src)),
         o_cp = take(bytes_of(C.cp)), o_cpp = take(bytes_of(C.cp_pred)),
         o_pp = take(bytes_of(C.pred_ptr)), o_pr = take(bytes_of(C.pred)),
         o_topo = take(bytes_of(C.topo)), o_wpp = take(bytes_of(C.wp_ptr)),
         o_wp = take(bytes_of(C.wp)), o_wsp = take(bytes_of(C.ws_ptr)), o_ws = take(bytes_of(C.ws)),
         o_evops = take(bytes_of(C.ev_ops)), o_evsucc = take(bytes_of(C.ev_succ)),
         o_jinfo = take(bytes_of(C.jinfo)), o_evsrc = take(bytes_of(C.ev_src)),
         o_rec16 = take(bytes_of(C.ev_rec16)), o_lvl = take(bytes_of(C.lvl_of)),
         o_levend = take(bytes_of(C.levend));
  // attribution: predecessors by caller id (ascending; implied ones removed:
  // they finish strictly before the op that implies them) and resources
  std::vector<int32_t> ap_ptr(n_ops + 1, 0), ap, row_res(op_res, op_res + n_ops);
  {
    std::vector<std::vector<int32_t>> pl(n_ops);
    for (int32_t c = 0; c < n_ops; ++c)
      for (int32_t k = C.pred_ptr[c]; k < C.pred_ptr[c + 1]; ++k) pl[C.ops[c].orig].push_back(C.ops[C.pred[k]].orig);
    for (int32_t v = 0; v < n_ops; ++v) {
      std::sort(pl[v].begin(), pl[v].end());
      ap.insert(ap.end(), pl[v].begin(), pl[v].end());
      ap_ptr[v + 1] = (int32_t)ap.size();
    }
  }
  const size_t o_app = take(bytes_of(ap_ptr)), o_ap = take(bytes_of(ap)), o_rres = take(bytes_of(row_res));
  if (hipMalloc(&g->dev_mem, off ? off : 256) != hipSuccess) {
    delete g;
    return SIM_E_NOMEM;
  }
  char *base = (char *)g->dev_mem;
  auto put = [&](size_t o, const void *src, size_t b) {
    return b == 0 || hipMemcpy(base + o, src, b, hipMemcpyHostToDevice) == hipSuccess;
  };
  bool ok = put(o_ops, C.ops.data(), bytes_of(C.ops)) && put(o_succ, C.succ.data(), bytes_of(C.succ)) &&
            put(o_jneed, C.jneed.data(), bytes_of(C.jneed)) && put(o_src, C.src.data(), bytes_of(C.src)) &&
            put(o_cp, C.cp.data(), bytes_of(C.cp)) && put(o_cpp, C.cp_pred.data(), bytes_of(C.cp_pred)) &&
            put(o_pp, C.pred_ptr.data(), bytes_of(C.pred_ptr)) && put(o_pr, C.pred.data(), bytes_of(C.pred)) &&
            put(o_topo, C.topo.data(), bytes_of(C.topo)) &&
            put(o_wpp, C.wp_ptr.data(), bytes_of(C.wp_ptr)) && put(o_wp, C.wp.data(), bytes_of(C.wp)) &&
            put(o_wsp, C.ws_ptr.data(), bytes_of(C.ws_ptr)) && put(o_ws, C.ws.data(), bytes_of(C.ws)) &&
            put(o_app, ap_ptr.data(), bytes_of(ap_ptr)) && put(o_ap, ap.data(), bytes_of(ap)) &&
            put(o_rres, row_res.data(), bytes_of(row_res)) &&
            put(o_evops, C.ev_ops.data(), bytes_of(C.ev_ops)) && put(o_evsucc, C.ev_succ.data(), bytes_of(C.ev_succ)) &&
            put(o_jinfo, C.jinfo.data(), bytes_of(C.jinfo)) && put(o_evsrc, C.ev_src.data(), bytes_of(C.ev_src)) &&
            put(o_rec16, C.ev_rec16.data(), bytes_of(C.ev_rec16)) &&
            put(o_lvl, C.lvl_of.data(), bytes_of(C.lvl_of)) && put(o_levend, C.levend.data(), bytes_of(C.levend));
  if (!ok) {
    (void)hipFree(g->dev_mem);
    delete g;
    return SIM_E_HIP;
  }
  DevGraph &d = g->dg;
  d.n = n_ops;
  d.R = n_res;
  d.J = C.JS;
  d.nsrc = (int32_t)C.src.size();
  d.heap_cap = C.heap_cap;
  d.cp_slots = C.cp_slots;
  d.cp_n = C.cp_n;
  d.max_indeg = C.max_indeg;
  d.ops = (const OpRec *)(base + o_ops);
  d.succ = (const int32_t *)(base + o_succ);
  d.jneed = (const int32_t *)(base + o_jneed);
  d.src = (const int32_t *)(base + o_src);
  d.cp = (const CpRec *)(base + o_cp);
  d.cp_pred = (const int32_t *)(base + o_cpp);
  d.pred_ptr = (const int32_t *)(base + o_pp);
  d.pred = (const int32_t *)(base + o_pr);
  d.topo = (const int32_t *)(base + o_topo);
  d.nb = C.barriers;
  d.wp_ptr = (const int32_t *)(base + o_wpp);
  d.wp = (const int32_t *)(base + o_wp);
  d.ws_ptr = (const int32_t *)(base + o_wsp);
  d.ws = (const int32_t *)(base + o_ws);
  d.ap_ptr = (const int32_t *)(base + o_app);
  d.ap = (const int32_t *)(base + o_ap);
  d.row_res = (const int32_t *)(base + o_rres);
  d.ev_ops = (const OpRec *)(base + o_evops);
  d.ev_succ = (const int32_t *)(base + o_evsucc);
  d.jinfo = (const int2 *)(base + o_jinfo);
  d.ev_src = (const int32_t *)(base + o_evsrc);
  d.pk_sh = C.pk_sh;
  d.pk_join = C.pk_join;
  d.pk_jn = C.pk_jn;
  d.pk_jb = C.pk_jb;
  d.pk_rmask = (int32_t)((1u << C.pk_rb) - 1u);
  d.ev_compact = C.ev_compact;
  d.pk_rkey = C.pk_rkey;
  d.ev_rec16 = (const int4 *)(base + o_rec16);
  d.lvl_of = (const int32_t *)(base + o_lvl);
  d.levend = (const int32_t *)(base + o_levend);
  d.n_levels = C.levels;

  g->h_orig_of.resize(n_ops);
  for (int32_t c = 0; c < n_ops; ++c) g->h_orig_of[c] = C.ops[c].orig;
  g->n_barriers = C.barriers;
  g->row_identity = 1;
  for (int32_t c = 0; c < n_ops && g->row_identity; ++c) g->row_identity = C.ops[c].orig == c;
  g->h_pred_ptr = C.pred_ptr;
  g->h_pred = C.pred;
  g->h_res.assign(op_res, op_res + n_ops);

  rc = plan_scratch(g);
  if (!rc) rc = plan_share(g);
  if (!rc) rc = noalloc_setup(g->device);  // once per device, with it current
  if (rc) {
    sim_graph_destroy(g);
    return rc;
  }
  *out = g;
  return SIM_OK;
}

extern "C" void sim_graph_destroy(sim_graph *g) {
  if (!g) return;
  g->pool.destroy();
  g->sweep_pool.destroy();
  g->share_pool.destroy();
  if (g->dev_mem) (void)hipFree(g->dev_mem);
  delete g;
}

extern "C" int sim_testing_replan(sim_graph *g, int32_t what, int32_t value) {
  if (!g) return SIM_E_INVAL;
  Variant v = g->var;
  switch (what) {
    case SIM_TEST_AUTO: v = Variant{}; break;
    case SIM_TEST_EV_LDS_GROUPS:
      if (value < -1 || value > 8) return SIM_E_INVAL;
      v.ev_lds_groups = value;
      break;
    case SIM_TEST_EV_BLOCKS_CAP:
      if (value < 0) return SIM_E_INVAL;
      v.ev_blocks_cap = value;
      break;
    case SIM_TEST_EV_REG:
      if (value < -1 || value > 1) return SIM_E_INVAL;
      v.ev_reg = value;
      break;
    case SIM_TEST_CP_GLOBAL:
      if (value < 0 || value > 1) return SIM_E_INVAL;
      v.cp_global = value;
      break;
    case SIM_TEST_RF_GLOBAL:
      if (value < 0 || value > 1) return SIM_E_INVAL;
      v.rf_global = value;
      break;
    case SIM_TEST_SHARE_KEY_ID:
      if (value < 0 || value > 1) return SIM_E_INVAL;
      v.share_key_id = value;
      break;
    default: return SIM_E_INVAL;
  }
  // no call may be in flight: the old sets are freed
  if (hipDeviceSynchronize() != hipSuccess) return SIM_E_HIP;
  const bool share_again = v.share_key_id != g->var.share_key_id;
  g->var = v;
  if (int rc = plan_scratch(g)) return rc;
  return share_again ? plan_share(g) : SIM_OK;
}

extern "C" int sim_graph_info(const sim_graph *g, int32_t *n_ops, int32_t *n_res, int64_t *n_edges,
                              int32_t *n_joins, int32_t *n_levels) {
  if (!g) return SIM_E_INVAL;
  if (n_ops) *n_ops = g->n_ops;
  if (n_res) *n_res = g->n_res;
  if (n_edges) *n_edges = g->n_edges;
  if (n_joins) *n_joins = g->n_joins;
  if (n_levels) *n_levels = g->n_levels;
  return SIM_OK;
}

extern "C" const char *sim_strerror(int code) {
  switch (code) {
    case SIM_OK: return "success";
    case SIM_E_INVAL: return "invalid argument";
    case SIM_E_RANGE: return "index out of range";
    case SIM_E_CYCLE: return "graph has a cycle";
    case SIM_E_NOMEM: return "out of memory";
    case SIM_E_HIP: return "HIP runtime error";
    case SIM_E_LIMIT: return "graph exceeds a library limit";
    default: return "unknown error";
  }
}

extern "C" int sim_testing_join_slots(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                                      const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                                      int32_t *slot_of, int32_t *n_slots) {
  if (!n_slots || (n_ops > 0 && !slot_of)) return SIM_E_INVAL;
  if (int rc = check_graph_args(n_ops, n_res, succ_ptr, succ_idx, op_res)) return rc;
  try {
    Compiled C;
    if (int rc = compile(n_ops, n_res, succ_ptr, succ_idx, op_res, prio, C)) return rc;
    for (int32_t c = 0; c < n_ops; ++c) {
      const int32_t j = C.join_of[c];
      slot_of[C.ops[c].orig] = j < 0 ? -1 : C.jslot[j];
    }
    *n_slots = C.JS;
  } catch (const std::bad_alloc &) {
    return SIM_E_NOMEM;
  }
  return SIM_OK;
}

extern "C" int sim_testing_sweep_table(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                                       const int32_t *succ_idx, const int32_t *op_res,
                                       const int32_t *prio, const int32_t *order, int32_t *n_rec,
                                       int32_t *slots, int32_t *rec, int64_t rec_cap, int32_t *plist,
                                       int64_t plist_cap, int64_t *plist_len) {
  if (!n_rec || !slots || !plist_len || rec_cap < 0 || plist_cap < 0) return SIM_E_INVAL;
  if ((rec_cap > 0 && !rec) || (plist_cap > 0 && !plist)) return SIM_E_INVAL;
  if (int rc = check_graph_args(n_ops, n_res, succ_ptr, succ_idx, op_res)) return rc;
  std::vector<CpRec> table;
  std::vector<int32_t> pl;
  int32_t ns = 0, sl = 0;
  try {
    Compiled C;
    if (int rc = compile(n_ops, n_res, succ_ptr, succ_idx, op_res, prio, C)) return rc;
    if (!order) {
      table = std::move(C.cp);
      pl = std::move(C.cp_pred);
      ns = C.cp_n;
      sl = C.cp_slots;
    } else {
      std::vector<int32_t> orig_of(n_ops);
      for (int32_t c = 0; c < n_ops; ++c) orig_of[c] = C.ops[c].orig;
      const std::vector<int32_t> res(op_res, op_res + n_ops);
      if (int rc = static_table(n_ops, orig_of, C.pred_ptr, C.pred, res, order, table, pl, sl, ns)) return rc;
    }
  } catch (const std::bad_alloc &) {
    return SIM_E_NOMEM;
  }
  *n_rec = ns;
  *slots = sl;
  *plist_len = (int64_t)pl.size();
  if (ns > rec_cap || (int64_t)pl.size() > plist_cap) return SIM_E_LIMIT;
  for (int32_t k = 0; k < ns; ++k) {
    const CpRec &r = table[k];
    const int32_t w[8] = {r.orig, r.slot, r.npred, r.pbeg, r.p[0], r.p[1], r.p[2], r.p[3]};
    std::memcpy(rec + 8 * (size_t)k, w, sizeof w);
  }
  if (!pl.empty()) std::memcpy(plist, pl.data(), pl.size() * 4);
  return SIM_OK;
}
