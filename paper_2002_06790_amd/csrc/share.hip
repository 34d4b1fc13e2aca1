// gfx950 kernel of the replay with bandwidth sharing: on a shared resource
// (a link) every op that becomes ready starts at once and the active ops
// divide its rate equally (processor sharing; the paper leaves concurrent
// transfers sharing one link's bandwidth to future work, Sec. 4).
//
// Model, in integer ns.  Between two consecutive event times t1 < t2 every
// active op of a shared resource with k active ops receives
// (t2 - t1) * floor(kShareUnit / k) service units (kShareUnit =
// 2^12 lcm(1..16): an exact equal share whenever k divides it).  The resource
// keeps the units one op has received since time 0 (vt, as of time tl); an
// op that arrives at time a with duration d needs vt(a) + d * kShareUnit and
// leaves at the first integer ns t with vt(t) >= that.  Finishes on shared
// resources at time t come before ready ops keyed t (lower resource first);
// ready ops keep the (ready time, priority, id) order of the plain replay,
// and other resources run their queues first in first out as there.
//
// Layout.  One scenario per lane.  A lane's event list is a 4-ary heap in
// global scratch of 64-bit keys (time << 32 | word), word = resource for a
// pending finish on a shared resource and n_res + compact id for a ready
// op (with the op's resource in the low bits below the id when it fits, so
// a popped op's resource state is requested together with its record), so
// one key order gives all the tie rules above.  The next finish of a
// shared resource changes when an op arrives or leaves.  The heap holds one
// current key per busy shared resource, whose time (pk) is at most its next
// finish: a departure, or an arrival that moves the next finish earlier,
// pushes a new key (an older one is then skipped when popped); an arrival
// that moves it later pushes nothing, and when the held key comes up before
// the finish it is pushed again at the finish.  So a call's heap holds at
// most one key per ready op and two per op on a shared resource.  The
// heap's top three levels (21 positions, 10.5 KB) live in LDS, the rest and
// all other per-lane state in global scratch, lane-major ([index][64]),
// except each shared resource's active ops, which a departure scans in
// order and so lie contiguous per lane: the {ready time, count} word of
// each node with two or more predecessors (a node with one predecessor is
// ready when it finishes and needs none), each resource's free time, each
// shared resource's 32-byte state record and its active ops.
#include <algorithm>
#include <cstring>
#include <vector>

#include "sim.hpp"

namespace mlsim {

namespace {

constexpr uint32_t kI32Max = 0x7fffffffu;
constexpr uint32_t kNoTime = 0xffffffffu;
constexpr int64_t kShareHeapLds = 21;    // heap positions per lane in LDS: the top three levels (10.5 KB per wavefront)
constexpr int64_t kShareFlagsLds = 1024; // resource flags in LDS (4 KB) up to this many resources
// a pop reads a child group 4i + 1 .. 4i + 4 from LDS when it starts there,
// so no group may straddle the end of the LDS part (a smaller heap, whose
// positions from its capacity on are all empty, needs no such care)
static_assert(kShareHeapLds % 4 == 1, "the LDS part of the heap must end at a child group boundary");

struct ShArgs {
  int64_t n_scen;
  const int32_t *dur;
  int64_t ld_dur;
  int32_t *makespan;
  int32_t *finish;  // [n_ops][ld_fin] or null
  int64_t ld_fin;
  int32_t *status;
  const int32_t *share;  // [R] 0 / 1
  char *scratch;         // per block: the regions below
  int64_t block_bytes;
  int64_t heap_cap;      // heap entries per lane (keys present at once)
  int64_t max_keys;      // keys pushed over a whole replay (bounds its pops)
  int heap_lds;          // heap positions per lane kept in LDS (the top of the heap)
  int flags_lds;         // the resource flags are copied to LDS after the heap
  int rows_identity;     // compact ids equal the caller's op ids (duration rows)
  const int32_t *np_of;  // [n_slots] predecessors of each node with two or more
  const struct ShRec *rec;  // [n] per op
  const int2 *sent;      // successor entries of every op (see ShRec)
  const int32_t *mword;  // key words of barrier members, indexed like the node successor lists
  const int32_t *srcw;   // [nsrc] key words of the sources
  int kres, rb;          // ready-op key words hold the resource in their low rb bits
  int32_t n_slots;
  int64_t o_rc, o_rf, o_ln, o_need, o_op;  // byte offsets in a block's region
};

// One op of the sharing replay (32 bytes): its duration row, its resource,
// and its successor entries {key word of the node, the node's ready/count
// word slot or -1}, the first two inline (kShNone: none) and all of them at
// sent[eb ...].  A node's key word is n_res + (id << rb | resource) for an op
// (n_res + id when the resource does not fit), or -(x + 1) for a barrier
// node x, whose members' key words are mword[ws_ptr[x] .. ws_ptr[x + 1]).
constexpr int32_t kShNone = INT32_MIN;
struct __attribute__((aligned(16))) ShRec {
  int32_t orig, res, eb, ne;
  int32_t w0, s0, w1, s1;
};

// one shared resource's state in one lane: service units per active op
// since time 0 (vt, as of time tl), the least need of its active ops (mn),
// its pending finish time (nd), active count (k) and the time of the key
// the heap holds for it (pk <= nd; kNoTime: none); read and written whole
struct __attribute__((aligned(16))) LinkSt {
  uint64_t vt, mn;
  uint32_t tl, nd;
  int32_t k;
  uint32_t pk;
};

// Read-only tables read at wave-uniform indices: through the constant
// address space such reads become scalar loads.
template <class T>
using cptr = const __attribute__((address_space(4))) T *;
template <class T>
__device__ __forceinline__ cptr<T> as_const(const T *p) {
  return (cptr<T>)p;
}

// A loaded value consumed by an empty asm: a load in one branch of an
// LDS-or-global choice then differs from the other branch's, so the two are
// not merged into one generic-address (flat) load through a selected pointer.
template <class T>
__device__ __forceinline__ T sh_settle(T v) {
  asm volatile("" : "+v"(v));
  return v;
}

template <class T>
struct Lane {  // element i of a lane-major array
  T *p;
  __device__ __forceinline__ T &operator[](int64_t i) const { return p[i * kWave]; }
};

__global__ __launch_bounds__(kWave) void k_share(DevGraph G, ShArgs a) {
  extern __shared__ uint64_t lds_heap[];
  const int lane = threadIdx.x;
  const int n = G.n, R = G.R;
  char *blk = a.scratch + (int64_t)blockIdx.x * a.block_bytes;
  const Lane<uint64_t> heap_g{(uint64_t *)blk + lane};
  // heap position i: in LDS below heap_lds, else in global scratch
  const int64_t HL = a.heap_lds;
  // (each branch keeps its own instruction: LDS or global, never flat)
  auto hget = [&](int64_t i) -> uint64_t {
    if (i < HL) return lds_heap[i * kWave + lane];
    return sh_settle(heap_g[i]);
  };
  auto hset = [&](int64_t i, uint64_t v) {
    if (i < HL) {
      lds_heap[i * kWave + lane] = v;
    } else {
      heap_g[i] = v;
      asm volatile("" ::: "memory");
    }
  };
  int32_t *flags_l = (int32_t *)(lds_heap + HL * kWave);
  if (a.flags_lds) {
    for (int r = lane; r < R; r += kWave) flags_l[r] = a.share[r];
    __syncthreads();
  }
  // resource r shared?  (the LDS copy or the argument, each by its own load)
  auto shared_res = [&](int r) -> bool { return (a.flags_lds ? flags_l[r] : sh_settle(a.share[r])) != 0; };
  // per node with two or more predecessors: ready time (high word) and
  // predecessors not yet finished
  const Lane<uint64_t> rc{(uint64_t *)(blk + a.o_rc) + lane};
  const Lane<uint32_t> rf{(uint32_t *)(blk + a.o_rf) + lane};
  const Lane<LinkSt> lk{(LinkSt *)(blk + a.o_ln) + lane};
  // each shared resource's active ops: the service units each needs and its
  // compact id, [R][kShareMax] contiguous per lane (a departure scans a
  // resource's entries in order)
  uint64_t *const need = (uint64_t *)(blk + a.o_need) + (int64_t)lane * R * kShareMax;
  int32_t *const eop = (int32_t *)(blk + a.o_op) + (int64_t)lane * R * kShareMax;

  for (int64_t tile = blockIdx.x; tile * kWave < a.n_scen; tile += gridDim.x) {
    const int64_t s = tile * kWave + lane;
    if (s >= a.n_scen) continue;
    // any duration below 1 flags the scenario before its replay starts:
    // the whole column, sixteen rows requested at a time (coalesced across
    // the wave; row ids are uniform, read as scalars)
    uint32_t st = 0;
    {
      const cptr<OpRec> ops = as_const(G.ops);
      int32_t dmin = 1;
      for (int c0 = 0; c0 < n; c0 += 16) {
        int32_t x[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int c = c0 + j < n ? c0 + j : n - 1;
          const int row = a.rows_identity ? c : ops[c].orig;
          x[j] = a.dur[(int64_t)row * a.ld_dur + s];
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) dmin = x[j] < dmin ? x[j] : dmin;
      }
      if (dmin < 1) st |= SIM_ST_BAD_DUR;
    }
    uint32_t span = 0;
    if (!st) {
      // {ready 0, count} of every node with two or more predecessors
      const cptr<int32_t> np_of = as_const(a.np_of);
      for (int j0 = 0; j0 < a.n_slots; j0 += 8) {
        uint64_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (uint64_t)(uint32_t)np_of[j0 + j < a.n_slots ? j0 + j : j0];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (j0 + j < a.n_slots) rc[j0 + j] = v[j];
      }
      for (int r = 0; r < R; ++r) {
        rf[r] = 0;
        lk[r] = LinkSt{0, 0, 0, kNoTime, 0, kNoTime};
      }
      int64_t hs = 0;
      // a 4-ary heap: children of position i at 4i + 1 .. 4i + 4, whose keys
      // are requested together
      auto push = [&](uint64_t key) -> bool {
        if (hs >= a.heap_cap) return false;
        int64_t i = hs++;
        while (i > 0) {
          const int64_t p = (i - 1) >> 2;
          const uint64_t kp = hget(p);
          if (kp <= key) break;
          hset(i, kp);
          i = p;
        }
        hset(i, key);
        return true;
      };
      // remove the minimum (the caller read it): the last key sifted down
      auto pop_rest = [&]() {
        const uint64_t last = hget(--hs);
        int64_t i = 0;
        for (;;) {
          const int64_t l = 4 * i + 1;
          if (l >= hs) break;
          // the four children requested together (indices clamped into the
          // LDS part or the lane's region; positions from hs on are empty)
          uint64_t kc[4];
          if (l < HL) {
#pragma unroll
            for (int q = 0; q < 4; ++q) kc[q] = lds_heap[(l + q < HL ? l + q : HL - 1) * kWave + lane];
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) kc[q] = heap_g[l + q < a.heap_cap ? l + q : a.heap_cap - 1];
#pragma unroll
            for (int q = 0; q < 4; ++q) kc[q] = sh_settle(kc[q]);
          }
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (l + q >= hs) kc[q] = ~0ull;
          int64_t m = l;
          uint64_t km = kc[0];
#pragma unroll
          for (int q = 1; q < 4; ++q)
            if (kc[q] < km) {
              km = kc[q];
              m = l + q;
            }
          if (km >= last) break;
          hset(i, km);
          i = m;
        }
        if (hs > 0) hset(i, last);
      };
      auto key_of = [](uint32_t t, uint32_t w) -> uint64_t { return ((uint64_t)t << 32) | w; };
      bool ok = true;
      // a successor entry {key word w, word slot sl} of an op finished (or
      // whose outputs arrive) at t, sl's word already read (os): count the
      // predecessor and, when it was the last, push the node's key (a
      // barrier pushes its members: it is their only predecessor).  A node
      // with one predecessor is ready at t without touching a word.
      auto fire = [&](int32_t w, int32_t sl, uint64_t os, uint32_t t) {
        if (w == kShNone) return;
        uint32_t v = t;
        if (sl >= 0) {
          const uint32_t r0 = (uint32_t)(os >> 32);
          v = r0 > t ? r0 : t;
          const uint32_t left = (uint32_t)os - 1u;
          rc[sl] = ((uint64_t)v << 32) | left;
          if (left != 0) return;
        }
        if (w >= 0) {
          ok = ok && push(key_of(v, (uint32_t)w));
          return;
        }
        const int x = -w - 1;
        for (int e = G.ws_ptr[x]; e < G.ws_ptr[x + 1]; ++e) ok = ok && push(key_of(v, (uint32_t)a.mword[e]));
      };
      // every successor of an op (record halves A {row, resource, first
      // entry, entries} and B {entries 0 and 1}) at t: the words of the
      // inline entries requested together, the others four entries at a time
      // (the nodes of one list are distinct, so the words are independent)
      // (every load below reads a valid index, clamped where the entry is
      // absent, and its value is discarded afterwards: conditional loads
      // would each wait for their data before the next is issued)
      auto release_op = [&](const int4 A, const int4 B, uint32_t t) {
        const uint64_t o0 = rc[B.y >= 0 ? B.y : 0], o1 = rc[B.w >= 0 ? B.w : 0];
        fire(B.x, B.y, o0, t);
        fire(B.z, B.w, o1, t);
        for (int e = 2; e < A.w; e += 4) {
          int2 en[4];
          uint64_t os[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) en[j] = a.sent[A.z + (e + j < A.w ? e + j : e)];
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (e + j >= A.w) en[j] = make_int2(kShNone, -1);
#pragma unroll
          for (int j = 0; j < 4; ++j) os[j] = rc[en[j].y >= 0 ? en[j].y : 0];
#pragma unroll
          for (int j = 0; j < 4; ++j) fire(en[j].x, en[j].y, os[j], t);
        }
      };
      auto advance = [](LinkSt &L, uint32_t t) {
        if (L.k > 0) L.vt += (uint64_t)(t - L.tl) * (kShareUnit / (uint64_t)L.k);
        L.tl = t;
      };
      // the first integer ns at which the resource's next op (the one that
      // needs m units) is done, k > 0 ops active; saturated at 2^31 (a finish
      // there overflows)
      auto finish_at = [](const LinkSt &L, int k, uint64_t m) -> uint32_t {
        const uint64_t per_ns = kShareUnit / (uint64_t)k;
        const uint64_t dt = (m - L.vt + per_ns - 1) / per_ns;
        const uint64_t t = (uint64_t)L.tl + dt;
        return t > kI32Max ? kI32Max + 1u : (uint32_t)t;
      };
      const int4 *rec4 = (const int4 *)a.rec;
      const uint32_t rmask = (1u << a.rb) - 1u;
      for (int k = 0; k < G.nsrc; ++k) ok = ok && push(key_of(0, (uint32_t)a.srcw[k]));
      // every iteration pops one key and a replay pushes at most max_keys,
      // so the loop ends; the guard only bounds it explicitly
      for (int64_t it = 0; hs > 0 && ok && it <= a.max_keys; ++it) {
        const uint64_t key = hget(0);
        const uint32_t t = (uint32_t)(key >> 32), w = (uint32_t)key;
        // The event's loads go out before the minimum is removed from the
        // heap (they read nothing the heap holds), so their round trip
        // overlaps the sift-down's: for a pending finish the resource's
        // state, for a ready op its record, its duration and (when the key
        // word names the resource) the resource's state.
        const bool lnk = w < (uint32_t)R;
        const uint32_t u = w - (uint32_t)R;
        const int c = lnk ? 0 : a.kres ? (int)(u >> a.rb) : (int)u;
        int4 A = make_int4(0, 0, 0, 0), B = A;
        int32_t d = 0;
        int r = lnk ? (int)w : 0;
        bool shr = lnk;
        LinkSt L{};
        uint32_t rfree = 0;
        if (lnk) {
          L = lk[r];
        } else {
          A = rec4[2 * c];
          B = rec4[2 * c + 1];
          if (a.rows_identity) d = a.dur[(int64_t)c * a.ld_dur + s];
          if (a.kres) {
            r = (int)(u & rmask);
            shr = shared_res(r);
            if (shr)
              L = lk[r];
            else
              rfree = rf[r];
          }
        }
        pop_rest();
        if (lnk) {  // a pending finish on shared resource r
          if (L.k == 0 || L.pk != t) continue;  // superseded
          if (L.nd != t) {  // arrivals since moved the next finish later: key it now
            L.pk = L.nd;
            ok = ok && push(key_of(L.nd, (uint32_t)r));
            lk[r] = L;
            continue;
          }
          if (t > kI32Max) {
            st |= SIM_ST_OVERFLOW;
            break;
          }
          advance(L, t);
          int k = L.k;
          const uint64_t v_now = L.vt;
          const int64_t base = (int64_t)r * kShareMax;
          // which active ops have their units (bit i: entry i), and the
          // least need of the others; eight entries (and their ops)
          // requested at a time (entries from k on are in bounds and ignored)
          uint64_t gone = 0, m_rest = ~0ull;
          for (int i0 = 0; i0 < k; i0 += 8) {
            uint64_t x[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = need[base + i0 + j];
#pragma unroll
            for (int j = 0; j < 8; ++j)
              if (i0 + j < k) {
                if (x[j] <= v_now)
                  gone |= 1ull << (i0 + j);
                else
                  m_rest = x[j] < m_rest ? x[j] : m_rest;
              }
          }
          if (gone == 0) {  // cannot happen: the finish time was computed to complete an op
            ok = false;
            break;
          }
          // remove them from the highest entry down, moving the last entry
          // into each hole (entries above the hole are staying ones)
          while (gone) {
            const int i = 63 - __builtin_clzll(gone);
            gone &= ~(1ull << i);
            const int c = eop[base + i];
            if (i != k - 1) {
              need[base + i] = need[base + k - 1];
              eop[base + i] = eop[base + k - 1];
            }
            --k;
            const int4 A = rec4[2 * c], B = rec4[2 * c + 1];
            if (a.finish) a.finish[(int64_t)A.x * a.ld_fin + s] = (int32_t)t;
            span = t > span ? t : span;
            release_op(A, B, t);
          }
          L.k = k;
          if (k > 0) {
            L.mn = m_rest;
            L.nd = L.pk = finish_at(L, k, m_rest);
            ok = ok && push(key_of(L.nd, (uint32_t)r));
          } else {
            L.nd = L.pk = kNoTime;
          }
          lk[r] = L;
          continue;
        }
        // a ready op (its resource from the record when the key word has
        // no room for it)
        if (!a.kres) {
          r = A.y;
          shr = shared_res(r);
          if (shr)
            L = lk[r];
          else
            rfree = rf[r];
        }
        if (!a.rows_identity) d = a.dur[(int64_t)A.x * a.ld_dur + s];
        if (shr) {  // joins the resource's active ops at its ready time
          const int k = L.k;
          if (k == kShareMax) {
            st |= SIM_ST_SHARE_LIMIT;
            break;
          }
          advance(L, t);
          const uint64_t nv = L.vt + (uint64_t)d * kShareUnit;
          need[(int64_t)r * kShareMax + k] = nv;
          eop[(int64_t)r * kShareMax + k] = c;
          L.k = k + 1;
          L.mn = k == 0 || nv < L.mn ? nv : L.mn;
          L.nd = finish_at(L, k + 1, L.mn);
          // a new key only when the next finish moved earlier than the key
          // held; a later one is keyed when the held key comes up
          if (L.nd < L.pk) {
            L.pk = L.nd;
            ok = ok && push(key_of(L.nd, (uint32_t)r));
          }
          lk[r] = L;
          continue;
        }
        const uint32_t start = t > rfree ? t : rfree;
        const uint32_t f = start + (uint32_t)d;  // both terms <= INT32_MAX
        if (f > kI32Max) {
          st |= SIM_ST_OVERFLOW;
          break;
        }
        rf[r] = f;
        span = f > span ? f : span;
        if (a.finish) a.finish[(int64_t)A.x * a.ld_fin + s] = (int32_t)f;
        release_op(A, B, f);
      }
      if (!ok) st |= SIM_ST_INTERNAL;
    }
    a.makespan[s] = st ? -1 : (int32_t)span;
    if (a.status) a.status[s] = (int32_t)st;
  }
}

}  // namespace

namespace {
int64_t al256(int64_t b) { return (b + 255) & ~(int64_t)255; }

// bytes of one block's region for a heap of cap entries per lane (and the
// offsets of its parts in a)
int64_t share_block_bytes(int64_t R, int64_t cap, int64_t slots, ShArgs *a) {
  int64_t off = 0;
  off += al256(cap * 8 * kWave);
  if (a) a->o_rc = off;
  off += al256(std::max<int64_t>(slots, 1) * 8 * kWave);
  if (a) a->o_rf = off;
  off += al256(R * 4 * kWave);
  if (a) a->o_ln = off;
  off += al256(R * (int64_t)sizeof(LinkSt) * kWave);
  if (a) a->o_need = off;
  off += al256(R * kShareMax * 8 * kWave);
  if (a) a->o_op = off;
  off += al256(R * kShareMax * 4 * kWave);
  return off;
}

// a set's constant head after the resource flags: the graph tables
int fill_share_set(void *ctx, char *b) {
  const sim_graph *g = (const sim_graph *)ctx;
  const int64_t R = g->dg.R;
  if (!g->share_tables.empty() && hipMemcpy(b + al256(R * 4), g->share_tables.data(), g->share_tables.size(),
                                            hipMemcpyHostToDevice) != hipSuccess)
    return SIM_E_HIP;
  return SIM_OK;
}
}  // namespace

// Sized once per graph: the tables of the replay (the predecessor count of
// each node with two or more predecessors, per op its record and successor
// entries, the key words of barrier members and of sources), and one set
// holding the resource flags, the tables and the block regions, sized for
// the largest heap any call can need (every resource shared) within the
// budget.  When the device cannot hold the budget, fewer block regions are
// kept (a call then runs fewer blocks at a time).
int plan_share(sim_graph *g) {
  const DevGraph &G = g->dg;
  const int64_t n = G.n, N = (int64_t)G.n + G.nb, R = G.R;
  std::vector<int32_t> wp((size_t)N + 1), wsp((size_t)N + 1), src((size_t)G.nsrc);
  if (hipMemcpy(wp.data(), G.wp_ptr, wp.size() * 4, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(wsp.data(), G.ws_ptr, wsp.size() * 4, hipMemcpyDeviceToHost) != hipSuccess ||
      (G.nsrc && hipMemcpy(src.data(), G.src, src.size() * 4, hipMemcpyDeviceToHost) != hipSuccess))
    return SIM_E_HIP;
  std::vector<int32_t> ws((size_t)wsp[N]);
  if (!ws.empty() && hipMemcpy(ws.data(), G.ws, ws.size() * 4, hipMemcpyDeviceToHost) != hipSuccess)
    return SIM_E_HIP;
  // word slot of each node with two or more predecessors, and their counts
  std::vector<int32_t> slot_of((size_t)N, -1), np;
  for (int64_t x = 0; x < N; ++x)
    if (wp[x + 1] - wp[x] > 1) {
      slot_of[x] = (int32_t)np.size();
      np.push_back(wp[x + 1] - wp[x]);
    }
  g->share_slots = (int32_t)np.size();
  // key word of a ready op: n_res + (id << rb | resource) when that fits 32
  // bits, else n_res + id; a barrier node x is named -(x + 1)
  int32_t rb = 0;
  while ((1ll << rb) < R) ++rb;
  const bool kres = R + ((int64_t)n << rb) <= (int64_t)UINT32_MAX && !g->var.share_key_id;
  g->share_kres = kres;
  g->share_rb = kres ? rb : 0;
  auto res_of = [&](int64_t c) { return g->h_res[g->h_orig_of[c]]; };
  auto word = [&](int64_t x) -> int32_t {
    if (x >= n) return (int32_t)(-(x + 1));
    return (int32_t)(uint32_t)(R + (kres ? ((uint64_t)x << rb | (uint64_t)res_of(x)) : (uint64_t)x));
  };
  std::vector<ShRec> rec((size_t)n);
  std::vector<int2> sent;
  for (int64_t c = 0; c < n; ++c) {
    ShRec r{g->h_orig_of[c], res_of(c), (int32_t)sent.size(), wsp[c + 1] - wsp[c], kShNone, -1, kShNone, -1};
    for (int32_t e = wsp[c]; e < wsp[c + 1]; ++e) sent.push_back(make_int2(word(ws[e]), slot_of[ws[e]]));
    if (r.ne > 0) r.w0 = sent[r.eb].x, r.s0 = sent[r.eb].y;
    if (r.ne > 1) r.w1 = sent[r.eb + 1].x, r.s1 = sent[r.eb + 1].y;
    rec[c] = r;
  }
  std::vector<int32_t> mword(ws.size(), 0), srcw(src.size());
  for (int64_t x = n; x < N; ++x)  // barrier members (ops)
    for (int32_t e = wsp[x]; e < wsp[x + 1]; ++e) mword[e] = word(ws[e]);
  for (size_t k = 0; k < src.size(); ++k) srcw[k] = word(src[k]);
  // the tables, each 256-byte aligned, after the flags
  auto place = [](int64_t &off, int64_t bytes) {
    const int64_t o = off;
    off += al256(std::max<int64_t>(bytes, 4));
    return o;
  };
  int64_t off = 0;
  g->share_o_np = place(off, (int64_t)np.size() * 4);
  g->share_o_rec = place(off, (int64_t)rec.size() * (int64_t)sizeof(ShRec));
  g->share_o_sent = place(off, (int64_t)sent.size() * 8);
  g->share_o_mword = place(off, (int64_t)mword.size() * 4);
  g->share_o_srcw = place(off, (int64_t)srcw.size() * 4);
  g->share_tables.assign((size_t)off, 0);
  char *t = g->share_tables.data();
  if (!np.empty()) std::memcpy(t + g->share_o_np, np.data(), np.size() * 4);
  if (!rec.empty()) std::memcpy(t + g->share_o_rec, rec.data(), rec.size() * sizeof(ShRec));
  if (!sent.empty()) std::memcpy(t + g->share_o_sent, sent.data(), sent.size() * 8);
  if (!mword.empty()) std::memcpy(t + g->share_o_mword, mword.data(), mword.size() * 4);
  if (!srcw.empty()) std::memcpy(t + g->share_o_srcw, srcw.data(), srcw.size() * 4);
  const int64_t head = al256(R * 4) + off;
  const int64_t worst = share_block_bytes(R, (int64_t)G.heap_cap + 2 * (int64_t)G.n + 1, g->share_slots, nullptr);
  int64_t region = std::max(worst, std::min(kShareScratchBudget, kShareBlocksMax * worst));
  g->share_head = head;
  for (;;) {
    g->share_region = region;
    g->share_pool.destroy();
    const int rc = g->share_pool.init((size_t)(head + region), 1, false, fill_share_set, g);
    if (rc != SIM_E_NOMEM || region <= worst) return rc;
    (void)hipGetLastError();  // clear the failed allocation's error
    region = std::max(worst, region / 2);
  }
}

int launch_share(const sim_graph *g, char *b, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                 const int32_t *share_words, int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                 hipStream_t stream) {
  const DevGraph &G = g->dg;
  const int64_t R = G.R;
  // this call's heap: the ready ops not yet popped, which form an antichain
  // (a path between two of them would pass an unfinished predecessor), so
  // at most the minimum path cover of the DAG, plus two keys per op on a
  // shared resource (its arrival and at most one departure batch)
  int64_t m_sh = 0;
  for (int32_t v = 0; v < g->n_ops; ++v) m_sh += share_words[g->h_res[v]] != 0;
  const int64_t cap = (int64_t)G.heap_cap + 2 * m_sh + 1;
  ShArgs a{};
  a.block_bytes = share_block_bytes(R, cap, g->share_slots, &a);
  a.heap_cap = cap;
  a.max_keys = (int64_t)G.n + 2 * m_sh + 1;
  // LDS: the heap's top positions, then the resource flags when they are few
  a.flags_lds = R <= kShareFlagsLds;
  a.heap_lds = (int)std::min<int64_t>(cap, kShareHeapLds);
  a.rows_identity = g->row_identity;
  const size_t lds = (size_t)a.heap_lds * 8 * kWave + (a.flags_lds ? (size_t)R * 4 : 0);
  // the flags travel in stream order as kernel arguments, so the caller's
  // array is no longer read on return
  int32_t *flags = (int32_t *)b;
  if (int rc = launch_put_words(flags, share_words, (int32_t)R, stream)) return rc;
  // a persistent grid: as many blocks as the region holds, balanced so the
  // last round of tiles is not nearly empty
  const int64_t tiles = (n_scen + kWave - 1) / kWave;
  const int64_t fit = std::max<int64_t>(1, std::min<int64_t>(kShareBlocksMax, g->share_region / a.block_bytes));
  const int64_t rounds = (tiles + fit - 1) / fit;
  const int64_t blocks = std::min((tiles + rounds - 1) / rounds, fit);
  a.n_scen = n_scen;
  a.dur = dur;
  a.ld_dur = ld_dur;
  a.makespan = makespan;
  a.finish = finish;
  a.ld_fin = ld_fin;
  a.status = status;
  a.share = flags;
  const char *tab = b + al256(R * 4);
  a.np_of = (const int32_t *)(tab + g->share_o_np);
  a.rec = (const ShRec *)(tab + g->share_o_rec);
  a.sent = (const int2 *)(tab + g->share_o_sent);
  a.mword = (const int32_t *)(tab + g->share_o_mword);
  a.srcw = (const int32_t *)(tab + g->share_o_srcw);
  a.kres = g->share_kres;
  a.rb = g->share_rb;
  a.n_slots = g->share_slots;
  a.scratch = b + g->share_head;
  k_share<<<dim3((unsigned)blocks), dim3(kWave), lds, stream>>>(G, a);
  return hipGetLastError() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

}  // namespace mlsim
