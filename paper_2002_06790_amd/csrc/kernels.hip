// gfx950 kernels of the batched dataflow replay.
//
// Layout: one wavefront owns a tile of 64 consecutive scenarios, one scenario
// per lane.  Durations, placements and finish times are op-major x scenario,
// so a lane reads and writes its own column and lanes that touch the same op
// touch one contiguous 256-byte row.  Per-lane state is laid out slot-major x
// lane ([slot][64]) in LDS or in global scratch, so a wave's accesses to one
// slot index are conflict-free / coalesced.  A persistent grid strides over
// tiles; every kernel leaves its scratch in the state it found it.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "philox.hpp"
#include "regarr.hpp"
#include "sim.hpp"

namespace mlsim {

namespace {

constexpr uint32_t kI32Max = 0x7fffffffu;

// Graph tables are read-only for the whole launch.  Reading them through the
// constant address space lets wave-uniform reads become scalar loads.
template <class T>
using cptr = const __attribute__((address_space(4))) T *;
template <class T>
__device__ __forceinline__ cptr<T> as_const(const T *p) {
  return (cptr<T>)p;
}
__device__ __forceinline__ uint64_t make_key(uint32_t ready, int32_t c) {
  return ((uint64_t)ready << 32) | (uint32_t)c;
}

// LDS pointers carry their address space explicitly, so accesses compile to
// ds_* instructions and never to generic (flat) ones.
template <class T>
using lptr = __attribute__((address_space(3))) T *;
template <class T>
__device__ __forceinline__ lptr<T> as_lds(T *p) {
  return (lptr<T>)p;
}

// Wait for a global load inside the branch that issued it: the empty asm
// consumes the value, so the compiler's wait lands here and not at a later
// merge point, where it would also have to cover every load in flight.
template <class T>
__device__ __forceinline__ T settle(T v) {
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ int2 settle(int2 v) {
  asm volatile("" : "+v"(v.x), "+v"(v.y));
  return v;
}
__device__ __forceinline__ int4 settle(int4 v) {
  asm volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
  return v;
}

// Per-lane ready list: an 8-ary min-heap of 64-bit keys (ready << 32 |
// compact id).  Compact ids follow (priority, id), so key order is the queue
// order of a first-in-first-out resource with the tie rules.
//
// Positions run breadth-first from kRoot = 7, which puts the 8 children of
// position p at 8 (p - 6) ... 8 (p - 6) + 7: every child group is aligned to
// 8 entries.  The root is kept in a register, and with REG so are its 8
// children (an array read through selects only, so it stays in registers):
// that frees 4 KB of LDS per wavefront for more resident wavefronts at the
// price of some VALU work per step.  The next positions up to le - 1 (the
// children unless REG, then the first groups of the root's grandchildren,
// which breadth-first order fills first) live in LDS, slot-major x lane,
// conflict-free; positions from le on live in global scratch, lane-major, so
// one child group there is one aligned 64-byte segment of one lane.  Every
// position at or beyond the end holds kEmpty, which is larger than any key,
// so partial groups need no bounds masks; the kernel restores kEmpty
// wherever the heap shrinks, leaving scratch as it found it.
constexpr int kD = 8, kRoot = kD - 1, kL1 = kD, kL2 = 2 * kD;
constexpr uint64_t kEmpty = ~0ull;

__device__ __forceinline__ int heap_parent(int p) { return p / kD + (kRoot - 1); }
__device__ __forceinline__ int heap_child0(int p) { return kD * (p - (kRoot - 1)); }

template <bool REG>
struct WideHeap {
  static constexpr int kLB = REG ? kL2 : kL1;  // first heap position in LDS
  uint64_t root;     // position kRoot
  uint64_t ch[kD];   // REG: positions kL1 .. kL2 - 1, the root's children
  lptr<uint64_t> l;  // this lane's LDS column: position p (kLB .. le-1) at l[(p - kLB) * kWave]
  uint64_t *g;       // this lane's global run: position p (>= le) at g[p - le]
  int le;            // first position in global memory (kL2 + kD k)
  // child k of the root (k lane-dependent).  REG: a tree of selects on the
  // bits of k (a chain of equality selects would be turned back into an
  // indexed load, which would move the array to scratch memory)
  __device__ __forceinline__ uint64_t child(int k) const {
    if (!REG) return l[k * kWave];
    const bool b0 = k & 1, b1 = k & 2, b2 = k & 4;
    const uint64_t a01 = b0 ? ch[1] : ch[0], a23 = b0 ? ch[3] : ch[2];
    const uint64_t a45 = b0 ? ch[5] : ch[4], a67 = b0 ? ch[7] : ch[6];
    const uint64_t a03 = b1 ? a23 : a01, a47 = b1 ? a67 : a45;
    return b2 ? a47 : a03;
  }
  __device__ __forceinline__ void set_child(int k, uint64_t x) {
    if (!REG) {
      l[k * kWave] = x;
      return;
    }
#pragma unroll
    for (int j = 0; j < kD; ++j) ch[j] = k == j ? x : ch[j];
  }
  // all 8 children of the root
  __device__ __forceinline__ void children(uint64_t (&v)[kD]) const {
#pragma unroll
    for (int k = 0; k < kD; ++k) v[k] = REG ? ch[k] : l[k * kWave];
  }
  __device__ __forceinline__ uint64_t get(int p) const {
    if (REG && p < kL2) return child(p - kL1);
    if (p < le) return l[(p - kLB) * kWave];
    return settle(g[p - le]);
  }
  __device__ __forceinline__ void set(int p, uint64_t x) {
    if (REG && p < kL2)
      set_child(p - kL1, x);
    else if (p < le)
      l[(p - kLB) * kWave] = x;
    else
      g[p - le] = x;
  }
  // the group starting at c (kLB <= c < le, a multiple of kD) in LDS
  __device__ __forceinline__ void lds_group(int c, uint64_t (&v)[kD]) const {
#pragma unroll
    for (int k = 0; k < kD; ++k) v[k] = l[(c + k - kLB) * kWave];
  }
  // the group starting at c >= le: one aligned 64-byte segment
  __device__ __forceinline__ void global_group(int c, uint64_t (&v)[kD]) const {
    const uint4 *gp = (const uint4 *)(g + (c - le));
    uint4 w[kD / 2];
#pragma unroll
    for (int k = 0; k < kD / 2; ++k) w[k] = gp[k];
#pragma unroll
    for (int k = 0; k < kD / 2; ++k) {
      v[2 * k] = ((uint64_t)w[k].y << 32) | w[k].x;
      v[2 * k + 1] = ((uint64_t)w[k].w << 32) | w[k].z;
    }
  }
};

// Minimum of kD keys and its index, as a balanced tree (short dependency chain).
__device__ __forceinline__ void min_group(uint64_t (&v)[kD], uint64_t &m, int &q) {
  int ix[kD];
#pragma unroll
  for (int k = 0; k < kD; ++k) ix[k] = k;
#pragma unroll
  for (int st = 1; st < kD; st <<= 1)
#pragma unroll
    for (int k = 0; k < kD; k += 2 * st)
      if (v[k + st] < v[k]) {
        v[k] = v[k + st];
        ix[k] = ix[k + st];
      }
  m = v[0];
  q = ix[0];
}

// Place x at position p (a grandchild of the root or deeper) of a heap
// ending at `end` and restore heap order below it; every group below a
// grandchild of the root lies in global memory (one round trip per level).
template <class H>
__device__ __forceinline__ void sift_down_deep(H &h, int end, int p, uint64_t x) {
  for (;;) {
    const int c = heap_child0(p);
    if (c >= end) break;
    uint64_t v[kD], m;
    int q;
    h.global_group(c, v);
    min_group(v, m, q);
    if (x < m) break;  // keys are distinct; kEmpty is above every key
    h.set(p, m);
    p = c + q;
  }
  h.set(p, x);
}

// Append x and restore heap order above it.
template <class H>
__device__ __forceinline__ void heap_push(H &h, int &end, uint64_t x) {
  int p = end++;
  while (p > kRoot) {
    const int par = heap_parent(p);
    const uint64_t a = par == kRoot ? h.root : h.get(par);
    if (a < x) break;
    h.set(p, a);
    p = par;
  }
  if (p == kRoot)
    h.root = x;
  else
    h.set(p, x);
}

// What one replay step reads of its heap before it knows the new key: the
// smallest child of the root, that child's own child group and, when it sits
// in global memory and the kernel is not LAZY, the last element.  The global loads go out with the
// step's duration and record loads, so a sift-down costs no round trip of
// its own unless it goes deeper than the root's grandchildren.
struct HeapAhead {
  bool eager;       // the last element is requested with the look-ahead (else when a pop needs it)
  uint64_t m1;      // smallest child of the root (kEmpty if none)
  int q1;           // its position
  int c2;           // first child of q1 (>= end: none)
  uint64_t v2[kD];  // that group (valid if c2 < end)
  uint64_t m2;      // its minimum
  int q2;           // the minimum's index in the group
  uint64_t last;    // the last element when it sits in global memory (eager)
};

template <bool DEEP, class H>
__device__ __forceinline__ void heap_look_ahead(const H &h, int end, HeapAhead &A) {
  uint64_t v[kD];
  h.children(v);  // all kEmpty when the root has no children
  min_group(v, A.m1, A.q1);
  A.q1 += kL1;
  A.c2 = heap_child0(A.q1);
  A.last = kEmpty;
  if (DEEP) {
    if (A.c2 < end && A.c2 >= h.le) h.global_group(A.c2, A.v2);
    if (A.eager && end - 1 >= h.le) A.last = h.g[end - 1 - h.le];
  }
  if (A.c2 < end && A.c2 < h.le) h.lds_group(A.c2, A.v2);
}

// Use the look-ahead loads on every path (their minimum is needed on most),
// so no load is still in flight when the step ends: a wait at the top of the
// next step would also wait for this step's stores.  Lanes whose root child
// has no children compute a minimum of stale values that nothing reads.
template <bool DEEP>
__device__ __forceinline__ void heap_settle_ahead(HeapAhead &A) {
  // the empty asm pins the wait here: a plain use could be sunk into the
  // branch that needs the minimum, leaving the loads pending on the others
  uint64_t v[kD];
#pragma unroll
  for (int k = 0; k < kD; ++k) v[k] = A.v2[k] = DEEP ? settle(A.v2[k]) : A.v2[k];
  min_group(v, A.m2, A.q2);
  if (DEEP && A.eager) A.last = settle(A.last);
}

// Replace the root by x (the first op a step releases), using the look-ahead.
template <class H>
__device__ __forceinline__ void heap_replace_root(H &h, int end, const HeapAhead &A, uint64_t x) {
  if (x < A.m1) {  // also when the root has no children (m1 = kEmpty)
    h.root = x;
    return;
  }
  h.root = A.m1;
  const int p = A.q1;
  if (A.c2 >= end || x < A.m2) {
    h.set_child(p - kL1, x);
    return;
  }
  h.set_child(p - kL1, A.m2);
  sift_down_deep(h, end, A.c2 + A.q2, x);
}

// Remove the root when the step released nothing, using the look-ahead.
template <class H>
__device__ __forceinline__ void heap_pop_root(H &h, int &end, HeapAhead &A) {
  const int lp = --end;  // position of the last element
  if (lp == kRoot) {
    h.root = kEmpty;
    return;
  }
  uint64_t x;
  if (lp < kL2) {
    x = h.child(lp - kL1);
    h.set_child(lp - kL1, kEmpty);
  } else if (lp < h.le) {
    x = h.l[(lp - H::kLB) * kWave];
    h.l[(lp - H::kLB) * kWave] = kEmpty;
  } else {
    x = A.eager ? A.last : settle(h.g[lp - h.le]);
    h.g[lp - h.le] = kEmpty;
  }
  if (lp < kL2) {  // a child of the root left: rescan them (no grandchildren remain)
    uint64_t v[kD];
    h.children(v);
    min_group(v, A.m1, A.q1);
    A.q1 += kL1;
    A.c2 = heap_child0(A.q1);
  } else if (lp == A.c2 + A.q2) {  // the look-ahead group's minimum left it: find the next one
#pragma unroll
    for (int k = 0; k < kD; ++k)  // unrolled: no indexed register access
      if (k == A.q2) A.v2[k] = kEmpty;
    min_group(A.v2, A.m2, A.q2);
  }
  heap_replace_root(h, end, A, x);
}

struct EvArgs {
  int64_t n_scen;
  const int32_t *dur;
  int64_t ld_dur;
  const uint16_t *place;
  int64_t ld_place;
  int32_t *makespan;
  int32_t *finish;
  int64_t ld_fin;
  int32_t *status;
  uint64_t *heap_g;   // [blocks][64][heap_stride]: heap positions from heap_le on, lane-major
  int heap_stride;    // entries per lane (a multiple of 16)
  int heap_le;        // first heap position in global memory (16 + 8 k)
  int2 *join_g;       // [blocks][J][64] {predecessors finished, max finish}
  uint32_t *rfree_g;  // [blocks][R][64] when resource times are not in LDS
  int32_t *prev;      // [n_ops][ld_fin] (PREV): the op that ran before each op on its resource, -1: none
  int32_t *last_g;    // [blocks][R][64] (PREV, resource times not in LDS): last op run per resource
  int last16;         // PREV with resource times in LDS: the last-op table holds 16-bit rows (0xffff: none)
  DurGen gen;         // GEN: durations generated from a knob grid and counter-based noise
  // device model, or null: [2R] words, each resource's idle time between
  // consecutive ops (gap) and then the time from an op's finish until its
  // outputs reach its successors (output delay)
  const int32_t *dev;
  int dev_gap, dev_delay;  // which of the two halves apply (uniform)
};

// finish times buffered per lane before a store burst: sixteen where the
// registers allow it without costing occupancy and it measured faster (the
// register-children variants with loaded durations, also those recording
// predecessors: at most two wavefronts per SIMD either way), else eight
constexpr int kFinQ = 8, kFinQWide = 16;

// A lane's join state {predecessors finished, max finish} per join index, in
// global scratch ([J][64] int2).
struct JoinGlobal {
  int2 *p;
  __device__ __forceinline__ int2 get(int j) const { return p[(size_t)j * kWave]; }
  __device__ __forceinline__ void set(int j, int2 v) const { p[(size_t)j * kWave] = v; }
};
// One replay step of k_event (see there).  DEEP: some lane's heap reaches
// global memory, so the step reads its heap ahead.
template <bool DEEP, bool RF_LDS, bool ROW_ID, bool PLACE, bool PREV, bool GEN, bool LAZY, class Heap, class JPtr,
          class RfGet, class RfSet, class LastXchg, class Flush, int FQ>
__device__ __forceinline__ void event_step(const DevGraph &G, const EvArgs &a, Heap &heap,
                                           int &end, JPtr jst, int it, int64_t s,
                                           int64_t sc, const int32_t *brow, uint32_t s_lo,
                                           uint32_t s_hi, uint32_t &st,
                                           uint32_t &span,
                                           int32_t (&fq)[FQ], int32_t (&rq)[FQ],
                                           int32_t (&pq)[FQ], RfGet rf_get, RfSet rf_set,
                                           LastXchg last_xchg, Flush flush) {
  const int R = G.R;
  const int2 *succ = (const int2 *)G.ev_succ;
  const int4 *rec4 = (const int4 *)G.ev_ops;
  // the step's loads go out at a raised wave priority (lowered once they
  // are issued), so with several wavefronts per SIMD the one starting a
  // step gets its requests in flight before others issue arithmetic
  __builtin_amdgcn_s_setprio(2);
  const uint64_t key = heap.root;
  const uint32_t low = (uint32_t)key;  // key word: compact id, maybe resource and first join
  const int c = (int)(low >> G.pk_sh);
  const uint32_t ready = (uint32_t)(key >> 32);
  // every global load of the step is issued before the first is used.
  // ROW_ID: the compact record {entry 0, entry 1}; otherwise the record
  // {orig, res, sbeg, nsucc} and {entry 0, entry 1}
  int4 r0, r1 = make_int4(0, 0, 0, 0);
  if (ROW_ID) {
    r0 = G.ev_rec16[c];
  } else {
    r0 = rec4[2 * c];
    r1 = rec4[2 * c + 1];
  }
  int32_t d = 0;
  int rp = 0;
  if (ROW_ID) {
    d = GEN ? brow[c] : a.dur[(int64_t)c * a.ld_dur + sc];
    if (PLACE)
      rp = a.place[(int64_t)c * a.ld_place + sc];
    else if (!G.pk_rkey)
      rp = G.row_res[c];  // the key word has no room for the resource
  }
  // the first successor's join state, when the key word names the join:
  // read together with the record instead of after it
  const uint32_t jmask = (1u << G.pk_jb) - 1u;
  const int jf = (int)(low & jmask);
  int2 js0 = make_int2(0, 0), ji0 = make_int2(0, 0);
  if (G.pk_join && (uint32_t)jf != jmask) {
    js0 = jst.get(jf);
    if (!G.pk_jn) ji0 = G.jinfo[jf];
  }
  // LAZY: the heap's last element is read when a pop needs it instead of
  // with the look-ahead (most steps release an op and pop nothing, so the
  // early load is mostly wasted address work; it measured faster only in
  // the register-children kernel with loaded durations and no device model)
  HeapAhead A;
  A.eager = !LAZY;
  heap_look_ahead<DEEP>(heap, end, A);
  // keep the scheduler from sinking these loads below the first use of d
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_setprio(0);
  const int32_t row = ROW_ID ? c : r0.x;
  if (!ROW_ID) {
    d = GEN ? brow[row] : a.dur[(int64_t)row * a.ld_dur + sc];
    if (PLACE) rp = a.place[(int64_t)row * a.ld_place + sc];
  }
  if (GEN) d = gen_duration(d, s_lo, s_hi, (uint32_t)row, a.gen.key0, a.gen.key1, a.gen.noise);
  int r = PLACE ? rp : !ROW_ID ? r0.y : G.pk_rkey ? (int)((low >> G.pk_jb) & (uint32_t)G.pk_rmask) : rp;
  if (PLACE && r >= R) {
    st |= SIM_ST_BAD_RES;
    r = 0;
  }
  // the device model's gap and delay of the resource: a small table read
  // from global memory (cached), requested before the duration is used
  int32_t gapv = 0, dlyv = 0;
  if (a.dev_gap) gapv = a.dev[r];
  if (a.dev_delay) dlyv = a.dev[R + r];
  if (d < 1) {
    st |= SIM_ST_BAD_DUR;
    d = 1;
  }
  const uint32_t rf = rf_get(r);
  const uint32_t start = ready > rf ? ready : rf;
  uint32_t fin = start + (uint32_t)d;  // both terms <= INT32_MAX: no uint32 wrap
  if (fin > kI32Max) {
    st |= SIM_ST_OVERFLOW;
    fin = kI32Max;
  }
  // the resource can start its next op at fin, or with gaps fin + gap[r];
  // successors see the outputs at fin, or with delays fin + delay[r] (both
  // saturated at 2^31, which still makes any later finish overflow)
  uint32_t avail = fin, out = fin;
  if (a.dev_gap) {
    const uint32_t x = fin + (uint32_t)gapv;
    avail = x < kI32Max + 1u ? x : kI32Max + 1u;
  }
  if (a.dev_delay) {
    const uint32_t x = fin + (uint32_t)dlyv;
    out = x < kI32Max + 1u ? x : kI32Max + 1u;
  }
  rf_set(r, avail);
  span = fin > span ? fin : span;
  const int32_t before = PREV ? last_xchg(r, row) : 0;  // the op this resource ran last
  heap_settle_ahead<DEEP>(A);
  // the record too: a step that releases nothing leaves its second half
  // unused, and a load still in flight at the end of a step makes the next
  // step wait for every store of this one before it can issue its loads
  const int4 r0s = settle(r0), r1s = ROW_ID ? r1 : settle(r1);
  // successor entries: the first two inline, the others (from index sbeg +
  // 2, or with ROW_ID from sbeg + 1) in the successor list
  int nsucc, sbeg;
  int2 e0, e1;
  bool more = false;
  if (ROW_ID) {
    e0 = make_int2(r0s.x, r0s.y);
    e1 = make_int2(r0s.z, r0s.w);
    more = e1.y < kRecNoSucc;
    nsucc = e0.y == kRecNoSucc ? 0 : e1.y == kRecNoSucc ? 1 : more ? 1 + (kRecMore - e1.y) : 2;
    sbeg = e1.x - 1;
  } else {
    e0 = make_int2(r1s.x, r1s.y);
    e1 = make_int2(r1s.z, r1s.w);
    nsucc = r0s.w;
    sbeg = r0s.z;
  }
  js0 = settle(js0);
  ji0 = settle(ji0);
  const int qs = it & (FQ - 1);  // wave-uniform
  if (!PLACE && !GEN) {
    // one indexed register move per array (the index is in a scalar register);
    // the placement and generated-duration kernels keep the compare chain,
    // which times faster there
    const int q = __builtin_amdgcn_readfirstlane(qs);
    fq[q] = (int32_t)fin;
    rq[q] = row;
    if (PREV) pq[q] = before;
  } else {
#pragma unroll
    for (int k = 0; k < FQ; ++k)
      if (k == qs) {
        fq[k] = (int32_t)fin;
        rq[k] = row;
        if (PREV) pq[k] = before;
      }
  }
  // a full burst goes out here, or for the placement kernels at the end of
  // the step (one counter covers loads and stores, so the loads of their
  // successor groups would wait behind it; the others measured faster here)
  if (!PLACE && qs == FQ - 1) flush(FQ);
  bool hole = true;  // the root was popped and is not yet replaced
  auto release = [&](uint32_t t, int w) {
    const uint64_t nk = make_key(t, w);
    if (hole) {
      heap_replace_root(heap, end, A, nk);
      hole = false;
    } else {
      heap_push(heap, end, nk);
    }
  };
  if (!PLACE) {
    for (int e = 0; e < nsucc; ++e) {
      const int2 sw = e == 0 ? e0 : e == 1 && !more ? e1 : settle(succ[sbeg + e]);  // {successor, join}
      if (sw.y < 0) {  // a plain successor, or the next member of a barrier
        release(sw.y == kJoinSibling ? ready : out, sw.x);
        continue;
      }
      // the join's state {predecessors finished, max finish} (already read for
      // the first entry when the key named it) and {predecessors needed, word
      // of the op released} (in the entry itself, or in the join table)
      const int j = G.pk_jn ? (sw.y & 0xffff) : sw.y;
      int2 js, ji;
      if (e == 0 && G.pk_join) {
        js = js0;
        ji = ji0;
      } else {
        js = settle(jst.get(j));
        if (!G.pk_jn) ji = settle(G.jinfo[j]);
      }
      if (G.pk_jn) ji = make_int2((int)((uint32_t)sw.y >> 16), sw.x);
      const uint32_t rdy = (uint32_t)js.y > out ? (uint32_t)js.y : out;
      if (js.x + 1 < ji.x) {
        jst.set(j, make_int2(js.x + 1, (int)rdy));
        continue;
      }
      jst.set(j, make_int2(0, 0));  // leave the join state clean
      // the join's op, or for a barrier its first member (the others follow it)
      release(rdy, ji.y);
    }
  } else {
    // one successor entry {successor, join} with its join's state js
    // {predecessors finished, max finish} and ji {predecessors needed, word of
    // the op released} (from the entry itself, or from the join table)
    auto handle = [&](int2 sw, int2 js, int2 ji) {
      if (sw.y < 0) {  // a plain successor, or the next member of a barrier
        release(sw.y == kJoinSibling ? ready : out, sw.x);
        return;
      }
      const int j = G.pk_jn ? (sw.y & 0xffff) : sw.y;
      if (G.pk_jn) ji = make_int2((int)((uint32_t)sw.y >> 16), sw.x);
      const uint32_t rdy = (uint32_t)js.y > out ? (uint32_t)js.y : out;
      if (js.x + 1 < ji.x) {
        jst.set(j, make_int2(js.x + 1, (int)rdy));
        return;
      }
      jst.set(j, make_int2(0, 0));  // leave the join state clean
      // the join's op, or for a barrier its first member (the others follow it)
      release(rdy, ji.y);
    };
    // The placement kernels take an op's first kC entries as one chunk: the
    // chunk's entries requested together, then their joins' states together,
    // two round trips in all instead of two per join.  Their ops release two
    // or three joins each, but the lanes of a wavefront pop different ops
    // and every lane waits for the one with the most entries (on random
    // layered graphs the largest of 64 lanes' counts is about eight: 4 and
    // 4 + 4 entries measured 10 % slower than 8, 12 and 16 slower too).
    // Entries beyond the chunk, rare, follow kC1 at a time.  Absent entries
    // load from clamped valid indices (one address, or one lane-major row,
    // across lanes) and are discarded; at one wavefront per CU they cost
    // little.  The successors of one op are distinct nodes whose joins never
    // share a slot, so none of these loads can see a store of the same op.
    // (The other kernels take one entry at a time, which needs fewer
    // registers and no wasted loads.)  The first chunk holds the inline
    // entries: e0 (its join's state already read with the record when the
    // key named it) and e1 (unless the record points to the list).
    constexpr int kC = 8, kC1 = 1;
    auto chunk = [&](auto first_tag, auto size_tag, int base) {
      constexpr bool F = decltype(first_tag)::value;
      constexpr int C = decltype(size_tag)::value;
      int2 sw[C], js[C], ji[C];
#pragma unroll
      for (int k = 0; k < C; ++k) {
        const int e = base + k;
        const bool inl = F && (k == 0 || (k == 1 && !more));
        const int2 m = succ[e < nsucc && !inl ? sbeg + e : 0];
        sw[k] = !F ? m : k == 0 ? e0 : k == 1 && !more ? e1 : m;
      }
#pragma unroll
      for (int k = 0; k < C; ++k) sw[k] = settle(sw[k]);
#pragma unroll
      for (int k = 0; k < C; ++k) {
        const bool first = F && k == 0 && G.pk_join;
        const bool joined = base + k < nsucc && sw[k].y >= 0 && !first;
        const int j = joined ? (G.pk_jn ? (sw[k].y & 0xffff) : sw[k].y) : 0;
        const int2 vs = G.J > 0 ? jst.get(j) : make_int2(0, 0);
        const int2 vi = G.J > 0 && !G.pk_jn ? G.jinfo[j] : make_int2(0, 0);
        js[k] = first ? js0 : vs;
        ji[k] = first ? ji0 : vi;
      }
#pragma unroll
      for (int k = 0; k < C; ++k) {
        js[k] = settle(js[k]);
        ji[k] = settle(ji[k]);
      }
#pragma unroll
      for (int k = 0; k < C; ++k)
        if (base + k < nsucc) handle(sw[k], js[k], ji[k]);
    };
    if (__ballot(nsucc > 0)) {  // some lane has entries
      chunk(std::true_type{}, std::integral_constant<int, kC>{}, 0);
      for (int base = kC; __ballot(base < nsucc); base += kC1)
        chunk(std::false_type{}, std::integral_constant<int, kC1>{}, base);
    }
  }
  if (hole) heap_pop_root(heap, end, A);
  if (PLACE && qs == FQ - 1) flush(FQ);
}

// Event-driven list scheduling, one scenario per lane (the paper's replay
// loop, Sec. 2).  Each lane keeps its ready list as a heap keyed by (ready
// time, compact id); it pops the minimum, starts it when both the op is ready
// and its resource has finished its previous op, and releases successors
// whose last predecessor this was.  Every lane pops exactly n ops per tile, so
// the outer loop is wave-uniform.  ROW_ID: the caller's op ids equal the
// compact ids, so the duration row is known as soon as the op is popped, and
// the graph has compact records (one 16-byte load per step; the resource
// comes from the key word, or when it has no room from a load by row issued
// with the record).
// PLACE: resources come from the per-scenario placement matrix.  Finish times
// are written in bursts of kFinQ (or kFinQWide) stores per lane, so their completion is
// waited for once per burst instead of once per step.  GEN: durations are
// generated from the knob grid and counter-based noise of a.gen instead of
// read from a.dur.  REG: the heap
// root's children live in registers (see WideHeap).  LAZY: the heap's last
// element is read only by steps that pop (see event_step).
template <bool RF_LDS, bool ROW_ID, bool PLACE, bool PREV, bool GEN = false, bool REG = false, bool LAZY = false>
__global__ __launch_bounds__(kWave) void k_event(DevGraph G, EvArgs a) {
  extern __shared__ uint64_t lds[];
  const int lane = threadIdx.x;
  const int n = G.n, R = G.R;
  WideHeap<REG> heap;
  heap.l = as_lds(lds) + lane;
  heap.g = a.heap_g + ((size_t)blockIdx.x * kWave + lane) * a.heap_stride;
  heap.le = a.heap_le;
  const int heap_lds = a.heap_le - WideHeap<REG>::kLB;  // heap positions per lane kept in LDS
  uint32_t *rfree_g = a.rfree_g + (size_t)blockIdx.x * R * kWave + lane;
  lptr<uint32_t> rfree_l = as_lds((uint32_t *)(lds + (size_t)heap_lds * kWave)) + lane;
  const JoinGlobal jst_g{a.join_g + (size_t)blockIdx.x * G.J * kWave + lane};
  auto rf_get = [&](int r) -> uint32_t { return RF_LDS ? rfree_l[r * kWave] : rfree_g[r * kWave]; };
  auto rf_set = [&](int r, uint32_t v) {
    if (RF_LDS)
      rfree_l[r * kWave] = v;
    else
      rfree_g[r * kWave] = v;
  };
  // PREV: the last op (row) each resource ran, next to the resource times
  // (in 16 bits when every row fits: half the LDS)
  lptr<int32_t> last_l = as_lds((int32_t *)(lds + (size_t)heap_lds * kWave) + (size_t)R * kWave) + lane;
  lptr<uint16_t> last_h = as_lds((uint16_t *)(lds + (size_t)heap_lds * kWave) + (size_t)2 * R * kWave) + lane;
  int32_t *last_g = PREV && !RF_LDS ? a.last_g + (size_t)blockIdx.x * R * kWave + lane : nullptr;
  auto last_xchg = [&](int r, int32_t row) -> int32_t {
    int32_t x;
    if (RF_LDS && a.last16) {
      const uint32_t h = last_h[r * kWave];
      x = h == 0xffffu ? -1 : (int32_t)h;
      last_h[r * kWave] = (uint16_t)row;
    } else if (RF_LDS) {
      x = last_l[r * kWave];
      last_l[r * kWave] = row;
    } else {
      x = last_g[r * kWave];
      last_g[r * kWave] = row;
    }
    return x;
  };

  for (int64_t tile = blockIdx.x; tile * kWave < a.n_scen; tile += gridDim.x) {
    const int64_t s = tile * kWave + lane;
    const bool active = s < a.n_scen;
    // the scenario column this lane replays (lanes past the end replay the last one)
    const int64_t sc = active ? s : a.n_scen - 1;
    const bool store_fin = a.finish && active;
    const int64_t S = GEN ? a.gen.scen0 + sc : 0;  // global scenario index of the generator
    const int32_t *brow = GEN ? gen_knob_row(a.gen, S) : nullptr;
    const uint32_t s_lo = (uint32_t)S, s_hi = (uint32_t)((uint64_t)S >> 32);
    for (int r = 0; r < R; ++r) rf_set(r, 0);
    if (PREV)
      for (int r = 0; r < R; ++r) {
        if (RF_LDS && a.last16)
          last_h[r * kWave] = 0xffffu;
        else if (RF_LDS)
          last_l[r * kWave] = -1;
        else
          last_g[r * kWave] = -1;
      }
    for (int k = 0; k < heap_lds; ++k) heap.l[k * kWave] = kEmpty;
    heap.root = kEmpty;
    if (REG)
#pragma unroll
      for (int k = 0; k < kD; ++k) heap.ch[k] = kEmpty;
    int end = kRoot;  // one past the last heap position
    for (int k = 0; k < G.nsrc; ++k) heap_push(heap, end, make_key(0, G.ev_src[k]));
    uint32_t st = 0, span = 0;
    constexpr int kQ = REG && !GEN ? kFinQWide : kFinQ;
    int32_t fq[kQ], rq[kQ], pq[kQ];  // buffered finish times, their rows, previous ops
    auto flush = [&](int cnt) {
#pragma unroll
      for (int k = 0; k < kQ; ++k)
        if (k < cnt && store_fin) {
          a.finish[(int64_t)rq[k] * a.ld_fin + s] = fq[k];
          if (PREV) a.prev[(int64_t)rq[k] * a.ld_fin + s] = pq[k];
        }
    };
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): the steps start with nothing in flight
    for (int it = 0; it < n; ++it) {
      if (end <= kRoot) break;  // unreachable for a DAG: some op is always ready
      auto run_step = [&](auto jp) {
        if (__ballot(end > heap.le))
          event_step<true, RF_LDS, ROW_ID, PLACE, PREV, GEN, LAZY>(G, a, heap, end, jp, it, s, sc, brow, s_lo, s_hi,
                                                             st, span, fq, rq, pq, rf_get, rf_set,
                                                             last_xchg, flush);
        else
          event_step<false, RF_LDS, ROW_ID, PLACE, PREV, GEN, LAZY>(G, a, heap, end, jp, it, s, sc, brow, s_lo,
                                                              s_hi, st, span, fq, rq, pq, rf_get, rf_set,
                                                              last_xchg, flush);
      };
      run_step(jst_g);
    }
    flush(n & (kQ - 1));
    if (st & (SIM_ST_BAD_DUR | SIM_ST_BAD_RES)) st &= ~(uint32_t)SIM_ST_OVERFLOW;
    if (active) {
      a.makespan[s] = st ? -1 : (int32_t)span;
      if (a.status) a.status[s] = (int32_t)st;
    }
  }
}

struct MpArgs {
  int64_t n_scen;
  const int32_t *dur;
  int64_t ld_dur;
  int32_t *out;       // [n_scen] longest path / makespan, -1 for a flagged scenario
  int32_t *status;    // [n_scen] status bits, or null
  int32_t *finish;    // [n_ops][ld_fin] dist of every op (FIN only)
  int64_t ld_fin;
  int32_t *dist_out;  // dist of every op (by caller id) for scenario dist_scen, or null
  int64_t dist_scen;
  uint32_t *slots_g;  // [blocks][slots][64] when slots are not in LDS
  DurGen gen;         // GEN: durations generated from a knob grid and counter-based noise
};

// Max-plus sweep, one scenario per lane: dist(v) = d(v) + max over v's
// predecessors in the table of their dist, in one topological order shared by
// the whole wave, in batches of kCpBatch records.  With the DAG's predecessors
// this is the longest path (critical path); with each op's previous op on its
// device added it is the static-order replay, whose dist is the finish time.
// A record is an op or a barrier node (row -1: duration 0, so its dist is the
// max over a predecessor set that several ops share, and those ops read it
// instead of the whole set).  Each op reads one coalesced duration row (and
// with FIN writes one finish row); dist of records that still have unvisited
// successors lives in value slots.  Software pipeline: while batch t is
// swept, the duration rows of batches t + 1 .. t + 3 and the records of batch
// t + 4 are in flight.  A batch's records arrive in two registers (lane i
// holds words i and 64 + i) and stay there until the batch is swept; a field
// is read by readlane, first the rows (for the batch's loads), later the rest
// (for its sweep).  MODE: where the value slots live (kCpSlotsLds or
// kCpSlotsGlobal); OUT: what besides the per-scenario result is written
// (kMpOutFinish: every op's dist as finish rows; kMpOutDist: every op's dist
// for one scenario).  GEN: a batch's "rows" are base durations of the lane's
// knob, and the sweep turns them into durations with the counter-based noise
// of a.gen.  BAR: the table holds barrier records.
template <int MODE, int OUT, bool GEN, bool BAR>
__global__ __launch_bounds__(kWave) void k_maxplus(MpTable T, MpArgs a) {
  extern __shared__ uint32_t lds32[];
  const int lane = threadIdx.x;
  const int n = T.n;
  constexpr int kRecWords = (int)(sizeof(CpRec) / 4);  // 8
  constexpr int kBatchWords = kCpBatch * kRecWords;    // 128: two words per lane
  static_assert(kBatchWords == 2 * kWave, "a batch of records is two words per lane");
  static_assert(kCpAhead == 4, "the pipeline below holds records four batches ahead");
  const int32_t *recw = (const int32_t *)T.rec;
  const cptr<int32_t> cp_pred = as_const(T.pred);
  uint32_t *slots = MODE == kCpSlotsLds ? lds32 + lane
                                        : a.slots_g + (size_t)blockIdx.x * T.slots * kWave + lane;
  auto sget = [&](int i) -> uint32_t { return slots[(size_t)i * kWave]; };
  auto sset = [&](int i, uint32_t x) { slots[(size_t)i * kWave] = x; };
  const int nbat = (n + kCpBatch - 1) / kCpBatch;
  sset(T.slots - 2, 0u);  // the slot that holds 0 (every other slot is written before it is read)
  for (int64_t tile = blockIdx.x; tile * kWave < a.n_scen; tile += gridDim.x) {
    const int64_t s = tile * kWave + lane;
    const bool active = s < a.n_scen;
    const int64_t sc = active ? s : a.n_scen - 1;
    const bool want_dist = OUT == kMpOutDist && s == a.dist_scen;
    const int64_t S = GEN ? a.gen.scen0 + sc : 0;  // global scenario index of the generator
    const int32_t *brow = GEN ? gen_knob_row(a.gen, S) : nullptr;
    const uint32_t s_lo = (uint32_t)S, s_hi = (uint32_t)((uint64_t)S >> 32);
    // The scenario is flagged at the end of its tile: a duration below 1
    // makes dmin < 1; a dist above INT32_MAX makes mx > INT32_MAX (the first
    // such dist is a sum of two terms <= INT32_MAX, so it does not wrap, and
    // mx never decreases).  A flagged scenario's dist values are unspecified,
    // so nothing is clamped on the way.
    uint32_t mx = 0;
    int32_t dmin = 1;
    struct Recs {
      int32_t w0, w1;  // lane i: words i and 64 + i of a batch's records
    };
    auto load_recs = [&](int t) -> Recs {
      return Recs{recw[(size_t)t * kBatchWords + lane], recw[(size_t)t * kBatchWords + kWave + lane]};
    };
    // rows of one batch (a barrier's row -1 reads row 0, which its sweep ignores)
    auto load_rows = [&](const Recs &r, int32_t (&dv)[kCpBatch]) {
#pragma unroll
      for (int u = 0; u < kCpBatch; ++u) {
        const int w = u * kRecWords;  // word of the batch holding the row
        const int32_t row = __builtin_amdgcn_readlane(w < kWave ? r.w0 : r.w1, w & (kWave - 1));
        const uint32_t rr = BAR && row < 0 ? 0u : (uint32_t)row;
        dv[u] = GEN ? brow[rr] : a.dur[(uint64_t)rr * (uint64_t)a.ld_dur + sc];
      }
    };
    auto sweep = [&](int t, const Recs &r, const int32_t (&dv)[kCpBatch]) {
#define CP_FIELD(u, f) __builtin_amdgcn_readlane(((u) * kRecWords + (f)) < kWave ? r.w0 : r.w1, ((u) * kRecWords + (f)) & (kWave - 1))
#pragma unroll
      for (int u = 0; u < kCpBatch; ++u) {
        // padding records (row of op 0, no predecessors, the sink slot) are
        // harmless to sweep unless they would write op 0's row
        if (OUT != kMpOutNone && t * kCpBatch + u >= n) break;
        const int np = CP_FIELD(u, 2);
        uint32_t best;
        if (__builtin_expect(np <= 4, 1)) {  // unused entries name the slot that holds 0
          const uint32_t x0 = sget(CP_FIELD(u, 4));
          const uint32_t x1 = sget(CP_FIELD(u, 5));
          const uint32_t x2 = sget(CP_FIELD(u, 6));
          const uint32_t x3 = sget(CP_FIELD(u, 7));
          const uint32_t m01 = x0 > x1 ? x0 : x1, m23 = x2 > x3 ? x2 : x3;
          best = m01 > m23 ? m01 : m23;
        } else {
          best = 0;
          const int pb = CP_FIELD(u, 3);
          for (int e = 0; e < np; ++e) {
            const uint32_t x = sget(cp_pred[pb + e]);
            best = x > best ? x : best;
          }
        }
        // A barrier's row -1 read op 0's durations (row 0, and op 0's noise
        // counter when generated), so dmin sees nothing that op 0 does not;
        // then a barrier adds 0 and writes no row.  No branch: a barrier's
        // dist never exceeds mx, the max of its predecessors' dist.
        const int32_t row = BAR || GEN || OUT != kMpOutNone ? CP_FIELD(u, 0) : 0;
        const int32_t keep = BAR ? ~(row >> 31) : -1;  // all ones for an op, 0 for a barrier
        int32_t d = dv[u];
        if (GEN) d = gen_duration(d, s_lo, s_hi, (uint32_t)(row & keep), a.gen.key0, a.gen.key1, a.gen.noise);
        dmin = d < dmin ? d : dmin;
        const uint32_t dist = best + (uint32_t)(d & keep);
        sset(CP_FIELD(u, 1), dist);
        mx = dist > mx ? dist : mx;
        if (OUT == kMpOutFinish && active && keep) a.finish[(int64_t)row * a.ld_fin + s] = (int32_t)dist;
        if (OUT == kMpOutDist && want_dist && keep) a.dist_out[row] = (int32_t)dist;
      }
#undef CP_FIELD
    };
    // One pipeline step: the records of batch t + 3 (loaded during step
    // t - 1, before batch t + 2's rows) give batch t + 3's rows; batch t + 4's
    // records go out; then batch t is swept.  Loads complete in issue order,
    // so waiting for the records leaves batch t + 2's rows in flight, and
    // waiting for batch t's rows leaves those of t + 1 .. t + 3 (48 row loads
    // and a record pair: within the 63 loads a wave can count).  r0 .. r2
    // hold the records of batches t .. t + 2, rx those of t + 3.
    Recs r0, r1, r2, rx;
    auto step = [&](int t, const int32_t (&cur)[kCpBatch], int32_t (&ahead3)[kCpBatch]) {
      const Recs r3 = rx;
      rx = load_recs(t + 4);
      load_rows(r3, ahead3);
      sweep(t, r0, cur);
      r0 = r1;
      r1 = r2;
      r2 = r3;
    };
    int32_t da[kCpBatch], db[kCpBatch], dc[kCpBatch], dd[kCpBatch];
    r0 = load_recs(0);
    r1 = load_recs(1);
    r2 = load_recs(2);
    load_rows(r0, da);
    load_rows(r1, db);
    rx = load_recs(3);
    load_rows(r2, dc);
    for (int t = 0; t < nbat; t += 4) {
      step(t, da, dd);
      if (t + 1 >= nbat) break;
      step(t + 1, db, da);
      if (t + 2 >= nbat) break;
      step(t + 2, dc, db);
      if (t + 3 >= nbat) break;
      step(t + 3, dd, dc);
    }
    const int32_t st = dmin < 1 ? SIM_ST_BAD_DUR : mx > kI32Max ? SIM_ST_OVERFLOW : 0;
    if (active) {
      a.out[s] = st ? -1 : (int32_t)mx;
      if (a.status) a.status[s] = st;
    }
  }
}

struct AtArgs {
  int64_t n_scen;
  const int32_t *dur;
  int64_t ld_dur;
  const uint16_t *place;
  int64_t ld_place;
  const int32_t *finish;  // [n_ops][ld_op] from the event replay
  const int32_t *prev;    // [n_ops][ld_op] each op's predecessor on its resource (-1: none)
  int64_t ld_op;
  const int32_t *status;  // [n_scen]
  int32_t *busy;          // [R][ld_res]
  int32_t *chain;         // [R][ld_res]
  int64_t ld_res;
  int32_t *chain_ops;     // [n_scen]
  uint32_t *acc_g;        // [blocks][2 R][64] when the accumulators are not in LDS
};

constexpr int kAtBatch = 8;  // rows loaded together in the busy-time sweep
constexpr int kAtPreds = 4;  // predecessor finish times loaded together in a chain step

// Bottleneck attribution, one scenario per lane (the paper's use of the
// simulator to find the bottleneck, Sec. 1).  First a sweep over all ops in
// id order (coalesced rows of durations and finish times) sums each
// resource's busy time and finds the op that finishes last (the lowest id
// among equals).  Then each lane walks its binding chain back from that op:
// from an op that starts at t > 0, to the lowest-id predecessor finishing at
// t if there is one, else to the op that ran before it on its resource; the
// walk ends at an op starting at 0 and adds each op's duration to its
// resource.  Scenarios with status bits get zeros and a chain length of -1.
template <bool PLACE, bool LDS>
__global__ __launch_bounds__(kWave) void k_attr(DevGraph G, AtArgs a) {
  extern __shared__ uint32_t lds32[];
  const int lane = threadIdx.x;
  const int n = G.n, R = G.R;
  uint32_t *busy_acc = LDS ? lds32 + lane : a.acc_g + (size_t)blockIdx.x * 2 * R * kWave + lane;
  uint32_t *chain_acc = busy_acc + (size_t)R * kWave;
  auto res_of = [&](int v, int64_t sc) -> int {
    return PLACE ? (int)a.place[(int64_t)v * a.ld_place + sc] : G.row_res[v];
  };
  for (int64_t tile = blockIdx.x; tile * kWave < a.n_scen; tile += gridDim.x) {
    const int64_t s = tile * kWave + lane;
    const bool active = s < a.n_scen;
    const int64_t sc = active ? s : a.n_scen - 1;
    const bool ok = active && a.status[s] == 0;
    for (int r = 0; r < R; ++r) {
      busy_acc[(size_t)r * kWave] = 0;
      chain_acc[(size_t)r * kWave] = 0;
    }
    uint32_t best = 0;
    int last = 0;
    for (int v0 = 0; v0 < n; v0 += kAtBatch) {
      int32_t dv[kAtBatch], fv[kAtBatch];
      int rv[kAtBatch];
#pragma unroll
      for (int u = 0; u < kAtBatch; ++u) {
        const int v = v0 + u < n ? v0 + u : n - 1;
        dv[u] = a.dur[(int64_t)v * a.ld_dur + sc];
        fv[u] = a.finish[(int64_t)v * a.ld_op + sc];
        rv[u] = res_of(v, sc);
      }
#pragma unroll
      for (int u = 0; u < kAtBatch; ++u) {
        if (v0 + u >= n) break;
        if ((unsigned)rv[u] < (unsigned)R) busy_acc[(size_t)rv[u] * kWave] += (uint32_t)dv[u];
        if ((uint32_t)fv[u] > best) {
          best = (uint32_t)fv[u];
          last = v0 + u;
        }
      }
    }
    // the binding chain (each op at most once: at most n steps)
    bool walking = ok;
    int v = last, ops = 0;
    for (int step = 0; step < n && __ballot(walking); ++step) {
      if (!walking) continue;
      const int32_t d = a.dur[(int64_t)v * a.ld_dur + s];
      const int32_t f = a.finish[(int64_t)v * a.ld_op + s];
      const int r = res_of(v, s);
      if ((unsigned)r < (unsigned)R) chain_acc[(size_t)r * kWave] += (uint32_t)d;
      ++ops;
      const int32_t start = f - d;
      if (start <= 0) {
        walking = false;
        continue;
      }
      int nxt = -1;
      for (int e0 = G.ap_ptr[v]; e0 < G.ap_ptr[v + 1] && nxt < 0; e0 += kAtPreds) {
        const int e1 = G.ap_ptr[v + 1];
        int pv[kAtPreds];
        int32_t fp[kAtPreds];
#pragma unroll
        for (int u = 0; u < kAtPreds; ++u) {
          pv[u] = G.ap[e0 + u < e1 ? e0 + u : e1 - 1];
          fp[u] = a.finish[(int64_t)pv[u] * a.ld_op + s];
        }
#pragma unroll
        for (int u = 0; u < kAtPreds; ++u)  // ascending ids: the first match is the lowest
          if (nxt < 0 && e0 + u < e1 && fp[u] == start) nxt = pv[u];
      }
      if (nxt < 0) nxt = a.prev[(int64_t)v * a.ld_op + s];
      if ((unsigned)nxt >= (unsigned)n)
        walking = false;  // cannot happen for a replay's own outputs
      else
        v = nxt;
    }
    if (active) {
      for (int r = 0; r < R; ++r) {
        a.busy[(int64_t)r * a.ld_res + s] = ok ? (int32_t)busy_acc[(size_t)r * kWave] : 0;
        a.chain[(int64_t)r * a.ld_res + s] = ok ? (int32_t)chain_acc[(size_t)r * kWave] : 0;
      }
      a.chain_ops[s] = ok ? ops : -1;
    }
  }
}

struct SwArgs {
  int64_t n_scen;
  const int32_t *dur;
  int64_t ld_dur;
  const uint16_t *place;
  int64_t ld_place;
  int32_t *makespan;
  int32_t *finish;
  int64_t ld_fin;
  int32_t *status;
  uint32_t *val_g;  // [blocks][n][64] per-op state when not in LDS
  uint32_t *res_g;  // [blocks][R][64] resource times, then [R][64] x2 uint64 bounds
};

constexpr uint32_t kDone = 0x80000000u;  // val bit: op committed (low bits: finish)

// Level-synchronous conservative sweeps, one scenario per lane.  A round
// first walks every uncommitted op in one topological order shared by the
// wave and computes lower bounds: est = max over predecessors of their finish
// (committed) or earliest finish (not committed), eft = max(est, resource
// free time) + d.  An op whose predecessors are all committed is ready at
// exactly est.  Then each resource commits its ready op of smallest key
// (est, compact id) if that key is below the bound of every op on the
// resource that is not ready yet.  Each resource therefore runs its ops in
// key order, which is the first-in-first-out replay's unique schedule; every
// round commits at least the globally smallest ready op.  The order is by
// level; a round sweeps from the first position some lane has not committed
// to the end of the level after the highest one committed, and bounds every
// op beyond it by one value (see below).
template <bool VAL_LDS, bool RES_LDS>
__global__ __launch_bounds__(kWave) void k_sweep(DevGraph G, SwArgs a) {
  extern __shared__ uint32_t sw_lds[];
  const int lane = threadIdx.x;
  const int n = G.n, R = G.R;
  uint32_t *val = VAL_LDS ? sw_lds + lane : a.val_g + (size_t)blockIdx.x * n * kWave + lane;
  uint32_t *resb = RES_LDS ? sw_lds + (VAL_LDS ? (size_t)n * kWave : 0)
                           : a.res_g + (size_t)blockIdx.x * R * kWave * 5;
  uint32_t *rfree = resb + lane;
  uint64_t *minf = (uint64_t *)(resb + (size_t)R * kWave) + lane;       // smallest ready key
  uint64_t *lbnd = (uint64_t *)(resb + (size_t)R * kWave * 3) + lane;   // smallest bound, not ready

  for (int64_t tile = blockIdx.x; tile * kWave < a.n_scen; tile += gridDim.x) {
    const int64_t s = tile * kWave + lane;
    const bool active = s < a.n_scen;
    const int64_t sc = active ? s : a.n_scen - 1;
    for (int v = 0; v < n; ++v) val[(size_t)v * kWave] = 0;
    for (int r = 0; r < R; ++r) rfree[r * kWave] = 0;
    int done = 0;
    uint32_t st = 0, span = 0;
    int lo = 0;       // positions before lo are committed in every lane
    int maxlc = -1;   // highest level this lane has committed
    for (int round = 0; round < n; ++round) {
      if (__ballot(done < n) == 0) break;
      for (int r = 0; r < R; ++r) {
        minf[r * kWave] = ~0ull;
        lbnd[r * kWave] = ~0ull;
      }
      while (lo < n && __ballot(!(val[(size_t)G.topo[lo] * kWave] & kDone)) == 0) ++lo;
      // An op can be ready only if its level is at most one above the
      // highest level committed, so positions past the end of that level
      // (highest over the wave) hold no ready op.  Every op there waits on a
      // chain of uncommitted ops that reaches the window, so its ready time
      // is at least bfar, the smallest earliest finish of an uncommitted op
      // in the window: one bound stands for all of them.
      int wl = maxlc;
#pragma unroll
      for (int off = kWave / 2; off > 0; off >>= 1) {
        const int o = __shfl_xor(wl, off);
        wl = o > wl ? o : wl;
      }
      const int hi = G.levend[wl + 1 < G.n_levels ? wl + 1 : G.n_levels - 1] + 1;
      uint32_t bfar = ~0u;
      for (int k = lo; k < hi; ++k) {
        const int v = G.topo[k];
        if (val[(size_t)v * kWave] & kDone) continue;
        uint32_t est = 0;
        bool ready = true;
        for (int e = G.pred_ptr[v]; e < G.pred_ptr[v + 1]; ++e) {
          const uint32_t y = val[(size_t)G.pred[e] * kWave];
          const uint32_t t = y & ~kDone;
          est = t > est ? t : est;
          ready = ready && (y & kDone);
        }
        const OpRec op = G.ops[v];
        int32_t d = a.dur[(int64_t)op.orig * a.ld_dur + sc];
        int r = op.res;
        if (a.place) {
          r = a.place[(int64_t)op.orig * a.ld_place + sc];
          if (r >= R) {
            st |= SIM_ST_BAD_RES;
            r = 0;
          }
        }
        if (d < 1) {
          st |= SIM_ST_BAD_DUR;
          d = 1;
        }
        const uint32_t rf = rfree[r * kWave];
        uint32_t eft = (est > rf ? est : rf) + (uint32_t)d;
        if (eft > kI32Max) eft = kI32Max;
        val[(size_t)v * kWave] = eft;
        bfar = eft < bfar ? eft : bfar;
        const uint64_t key = make_key(est, v);
        uint64_t *slot = ready ? &minf[r * kWave] : &lbnd[r * kWave];
        if (key < *slot) *slot = key;
      }
      // commit, per resource, the smallest ready op that beats every bound
      bool progress = false;
      uint64_t gmin = ~0ull;
      int gres = 0;
      for (int r = 0; r < R; ++r) {
        const uint64_t mf = minf[r * kWave];
        if (mf < gmin) {
          gmin = mf;
          gres = r;
        }
        if (mf < lbnd[r * kWave] && (uint32_t)(mf >> 32) < bfar) {
          progress = true;
          const int c = (int)(uint32_t)mf;
          const uint32_t rdy = (uint32_t)(mf >> 32);
          const OpRec op = G.ops[c];
          int32_t d = a.dur[(int64_t)op.orig * a.ld_dur + sc];
          d = d < 1 ? 1 : d;
          const uint32_t rf = rfree[r * kWave];
          uint32_t fin = (rdy > rf ? rdy : rf) + (uint32_t)d;
          if (fin > kI32Max) {
            st |= SIM_ST_OVERFLOW;
            fin = kI32Max;
          }
          rfree[r * kWave] = fin;
          val[(size_t)c * kWave] = fin | kDone;
          span = fin > span ? fin : span;
          ++done;
          maxlc = G.lvl_of[c] > maxlc ? G.lvl_of[c] : maxlc;
          if (a.finish && active) a.finish[(int64_t)op.orig * a.ld_fin + s] = (int32_t)fin;
        }
      }
      // Only saturated times (an overflowing scenario) can stall progress;
      // then commit the smallest ready op anyway so the sweep terminates.
      if (!progress && done < n && gmin != ~0ull) {
        const int c = (int)(uint32_t)gmin;
        const uint32_t rdy = (uint32_t)(gmin >> 32);
        const OpRec op = G.ops[c];
        int32_t d = a.dur[(int64_t)op.orig * a.ld_dur + sc];
        d = d < 1 ? 1 : d;
        const uint32_t rf = rfree[gres * kWave];
        uint32_t fin = (rdy > rf ? rdy : rf) + (uint32_t)d;
        if (fin > kI32Max) fin = kI32Max;
        st |= SIM_ST_OVERFLOW;
        rfree[gres * kWave] = fin;
        val[(size_t)c * kWave] = fin | kDone;
        ++done;
        maxlc = G.lvl_of[c] > maxlc ? G.lvl_of[c] : maxlc;
      }
    }
    if (st & (SIM_ST_BAD_DUR | SIM_ST_BAD_RES)) st &= ~(uint32_t)SIM_ST_OVERFLOW;
    if (active) {
      a.makespan[s] = st ? -1 : (int32_t)span;
      if (a.status) a.status[s] = (int32_t)st;
    }
  }
}

template <class K>
int occupancy_blocks(K kernel, size_t lds, int cus, bool strict = false) {
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kWave, lds) != hipSuccess)
    return -1;
  if (per_cu < 1) per_cu = strict ? 0 : 1;  // strict: 0 when the LDS does not fit one block
  return per_cu * cus;
}

constexpr size_t kRfLdsMax = 32 * 1024;        // resource times kept in LDS up to this size
constexpr size_t kScratchBudget = 4ull << 30;  // global per-block scratch of one kernel, per set
constexpr size_t kSweepBudget = 3ull << 30;    // the sweep variant's per-op state, per set of its own
constexpr size_t kPoolBudget = 4ull << 30;     // all eager sets of one graph together
constexpr int kMaxSets = 4;                    // eager sets per graph (at least one)

bool rf_in_lds(const sim_graph *g) {
  if (g->var.rf_global) return false;
  return (size_t)g->dg.R * kWave * 4 <= kRfLdsMax;
}

// a fresh set: join state cleared, heap positions empty (all ones); the
// kernels leave both that way
int fill_set(void *ctx, char *base) {
  const sim_graph *g = (const sim_graph *)ctx;
  if (hipMemset(base, 0, g->scratch_bytes) != hipSuccess) return SIM_E_HIP;
  if (g->heap_fill_bytes && hipMemset(base + g->scratch_ev_heap_off, 0xff, g->heap_fill_bytes) != hipSuccess)
    return SIM_E_HIP;
  return SIM_OK;
}

}  // namespace

int plan_scratch(sim_graph *g) {
  const DevGraph &G = g->dg;
  ScratchPlan &P = g->plan;
  const Variant &V = g->var;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, g->device) != hipSuccess) return SIM_E_HIP;
  const int cus = prop.multiProcessorCount;

  // event kernel: resource times in LDS when they fit; the root of each
  // lane's heap and its children in LDS, deeper positions (up to the exact
  // bound on ready ops) in global scratch
  const size_t rf_bytes = (size_t)G.R * kWave * 4;
  const bool rf_lds = rf_in_lds(g);
  P.rf_lds = rf_lds;
  P.ev_heap_stride = (int32_t)(((size_t)G.heap_cap + 2 * kD) & ~size_t(kD - 1));
  // groups of the root's grandchildren kept in LDS (4 KB per wave each):
  // four beside a small resource-time table, two beside a large one (heaps
  // of up to 41 or 25 entries then never touch global memory)
  const size_t rf_lds_bytes = rf_lds ? rf_bytes : 0;
  int lds_groups = rf_lds_bytes <= 8 * 1024 ? 4 : 2;
  if (V.ev_lds_groups >= 0) lds_groups = std::min(kD, V.ev_lds_groups);
  P.ev_heap_le = kL2 + kD * lds_groups;
  // join state in global scratch (in LDS it would cost more occupancy than
  // the round trip it saves: 45.4 vs 41.2 ms on the BERT workload)
  const size_t join_bytes = (size_t)G.J * kWave * 8;
  const size_t heap_g_bytes = (size_t)P.ev_heap_stride * kWave * 8;
  const size_t ev_per_block = join_bytes + heap_g_bytes + (rf_lds ? 0 : rf_bytes);
  auto grid_of = [&](int occ) -> int32_t {  // resident blocks within the scratch budget
    size_t b = (size_t)std::max(occ, 1);
    if (ev_per_block) b = std::min(b, std::max<size_t>(1, kScratchBudget / ev_per_block));
    if (V.ev_blocks_cap > 0) b = std::min(b, (size_t)V.ev_blocks_cap);
    return (int32_t)b;
  };
  // the root's children in LDS (every variant)
  P.ev_lds_bytes = (size_t)(P.ev_heap_le - kL1) * kWave * 8 + rf_lds_bytes;
  int occ[3];  // plain, generated durations, device model (its table is read from global memory)
  if (rf_lds) {
    occ[0] = occupancy_blocks(k_event<true, false, false, false>, P.ev_lds_bytes, cus);
    occ[1] = occupancy_blocks(k_event<true, false, false, false, true>, P.ev_lds_bytes, cus);
    occ[2] = occ[0];
  } else {
    occ[0] = occupancy_blocks(k_event<false, false, false, false>, P.ev_lds_bytes, cus);
    occ[1] = occupancy_blocks(k_event<false, false, false, false, true>, P.ev_lds_bytes, cus);
    occ[2] = occ[0];
  }
  if (occ[0] < 0 || occ[1] < 0 || occ[2] < 0) return SIM_E_HIP;
  P.ev_blocks = grid_of(occ[0]);
  P.ev_gen_blocks = grid_of(occ[1]);
  P.ev_dev_blocks = grid_of(occ[2]);
  // the root's children in registers (resource times in LDS, no placement,
  // no predecessor recording): 4 KB less LDS
  P.ev_reg = rf_lds;
  P.ev_reg_lds_bytes = (size_t)(P.ev_heap_le - kL2) * kWave * 8 + rf_lds_bytes;
  P.ev_reg_blocks = P.ev_reg_gen_blocks = P.ev_reg_dev_blocks = P.ev_reg_prev_blocks = 1;
  // the last-op table of attribution: 16-bit rows when every row fits
  P.ev_last16 = G.n < 0xffff;
  const size_t last_lds_bytes = P.ev_last16 ? rf_lds_bytes / 2 : rf_lds_bytes;
  P.ev_reg_prev_lds_bytes = P.ev_reg_lds_bytes + last_lds_bytes;  // with the last-op table
  if (P.ev_reg) {
    occ[0] = occupancy_blocks(k_event<true, false, false, false, false, true, true>, P.ev_reg_lds_bytes, cus);
    occ[1] = occupancy_blocks(k_event<true, false, false, false, true, true>, P.ev_reg_lds_bytes, cus);
    occ[2] = occupancy_blocks(k_event<true, false, false, false, false, true>, P.ev_reg_lds_bytes, cus);
    if (occ[0] < 0 || occ[1] < 0 || occ[2] < 0) return SIM_E_HIP;
    P.ev_reg_blocks = grid_of(occ[0]);
    P.ev_reg_gen_blocks = grid_of(occ[1]);
    P.ev_reg_dev_blocks = grid_of(occ[2]);
    const int prev_occ =
        occupancy_blocks(k_event<true, false, false, true, false, true>, P.ev_reg_prev_lds_bytes, cus);
    if (prev_occ < 0) return SIM_E_HIP;
    P.ev_reg_prev_blocks = grid_of(prev_occ);
  }
  // the event kernel for attribution: a last-op table beside the resource times
  P.ev_prev_lds_bytes = P.ev_lds_bytes + last_lds_bytes;
  const int ev_prev_occ = rf_lds ? occupancy_blocks(k_event<true, false, false, true>, P.ev_prev_lds_bytes, cus)
                                : occupancy_blocks(k_event<false, false, false, true>, P.ev_prev_lds_bytes, cus);
  if (ev_prev_occ < 0) return SIM_E_HIP;
  P.ev_prev_blocks = grid_of(ev_prev_occ);
  // A call with few tiles (fewer than the grids below hold) keeps the whole
  // third heap level in LDS: heaps of up to 73 entries then never touch
  // global memory.  Not planned when a test pins the LDS groups.
  P.ev_wide_le = kL2 + kD * kD;
  P.ev_wide_lds_bytes = (size_t)(P.ev_wide_le - kL1) * kWave * 8 + rf_lds_bytes;
  P.ev_wide_blocks = P.ev_wide_gen_blocks = P.ev_wide_dev_blocks = P.ev_wide_prev_blocks = 0;
  if (V.ev_lds_groups < 0 && lds_groups < kD) {
    const size_t wl = P.ev_wide_lds_bytes;
    int wo[4];
    if (rf_lds) {
      wo[0] = occupancy_blocks(k_event<true, false, false, false>, wl, cus, true);
      wo[1] = occupancy_blocks(k_event<true, false, false, false, true>, wl, cus, true);
      wo[2] = wo[0];
      wo[3] = occupancy_blocks(k_event<true, false, false, true>, wl + last_lds_bytes, cus, true);
    } else {
      wo[0] = occupancy_blocks(k_event<false, false, false, false>, wl, cus, true);
      wo[1] = occupancy_blocks(k_event<false, false, false, false, true>, wl, cus, true);
      wo[2] = wo[0];
      wo[3] = occupancy_blocks(k_event<false, false, false, true>, wl, cus, true);
    }
    if (wo[0] < 0 || wo[1] < 0 || wo[2] < 0 || wo[3] < 0) return SIM_E_HIP;
    auto wide_grid = [&](int occ) { return occ > 0 ? grid_of(occ) : 0; };  // 0: not available
    P.ev_wide_blocks = wide_grid(wo[0]);
    P.ev_wide_gen_blocks = wide_grid(wo[1]);
    P.ev_wide_dev_blocks = wide_grid(wo[2]);
    P.ev_wide_prev_blocks = wide_grid(wo[3]);
  }
  // attribution chains: busy and chain accumulators in LDS when they fit
  const size_t at_bytes = (size_t)2 * G.R * kWave * 4;
  P.at_lds = at_bytes <= 64 * 1024;
  P.at_lds_bytes = P.at_lds ? at_bytes : 8;
  const int at_occ = P.at_lds ? occupancy_blocks(k_attr<false, true>, P.at_lds_bytes, cus)
                              : occupancy_blocks(k_attr<false, false>, P.at_lds_bytes, cus);
  if (at_occ < 0) return SIM_E_HIP;
  P.at_blocks = (int32_t)(P.at_lds ? at_occ
                                   : std::min<size_t>(at_occ, std::max<size_t>(1, kScratchBudget / at_bytes)));

  // scratch for the largest persistent grid of any event variant
  const int32_t ev_grid = std::max({P.ev_blocks, P.ev_gen_blocks, P.ev_dev_blocks, P.ev_prev_blocks,
                                    P.ev_reg_blocks, P.ev_reg_gen_blocks, P.ev_reg_dev_blocks,
                                    P.ev_reg_prev_blocks, P.ev_wide_blocks, P.ev_wide_gen_blocks,
                                    P.ev_wide_dev_blocks, P.ev_wide_prev_blocks});

  // critical path: slots in LDS when they fit, else in global scratch
  const size_t cp_bytes = (size_t)G.cp_slots * kWave * 4;
  P.cp_mode = cp_bytes <= 32 * 1024 && !V.cp_global ? kCpSlotsLds : kCpSlotsGlobal;
  P.cp_lds_bytes = P.cp_mode == kCpSlotsLds ? cp_bytes : 0;
  const bool cp_bar = G.cp_n > G.n;
  const int cp_occ = maxplus_occupancy(P.cp_mode, false, P.cp_lds_bytes, cus, false, cp_bar);
  const int cp_gen_occ = maxplus_occupancy(P.cp_mode, false, P.cp_lds_bytes, cus, true, cp_bar);
  if (cp_occ < 0 || cp_gen_occ < 0) return SIM_E_HIP;
  size_t cp_blocks = (size_t)cp_occ;
  if (P.cp_mode == kCpSlotsGlobal && cp_bytes)
    cp_blocks = std::min(cp_blocks, std::max<size_t>(1, kScratchBudget / cp_bytes));
  P.cp_blocks = (int32_t)cp_blocks;
  P.cp_gen_blocks = (int32_t)std::min<size_t>(cp_blocks, (size_t)cp_gen_occ);
  // sweep variant: per-op state and per-resource state in LDS when small
  const size_t val_bytes = (size_t)G.n * kWave * 4;
  const size_t res_bytes = (size_t)G.R * kWave * 20;
  P.sw_val_lds = val_bytes <= 32 * 1024;
  P.sw_res_lds = res_bytes <= 16 * 1024;
  P.sw_lds_bytes = std::max<size_t>(8, (P.sw_val_lds ? val_bytes : 0) + (P.sw_res_lds ? res_bytes : 0));
  int sw_occ;
  if (P.sw_val_lds)
    sw_occ = P.sw_res_lds ? occupancy_blocks(k_sweep<true, true>, P.sw_lds_bytes, cus)
                          : occupancy_blocks(k_sweep<true, false>, P.sw_lds_bytes, cus);
  else
    sw_occ = P.sw_res_lds ? occupancy_blocks(k_sweep<false, true>, P.sw_lds_bytes, cus)
                          : occupancy_blocks(k_sweep<false, false>, P.sw_lds_bytes, cus);
  if (sw_occ < 0) return SIM_E_HIP;
  // the sweep's global state lives in sets of its own (one eager, one for
  // captures), as many blocks as kSweepBudget holds: it is latency-bound, so
  // its speed follows the resident blocks
  const size_t sw_val_blk = P.sw_val_lds ? 0 : (val_bytes + 255) & ~size_t(255);
  const size_t sw_res_blk = P.sw_res_lds ? 0 : (res_bytes + 255) & ~size_t(255);
  const size_t sw_per_block = sw_val_blk + sw_res_blk;
  size_t sw_blocks = (size_t)sw_occ;
  if (sw_per_block) sw_blocks = std::min(sw_blocks, std::max<size_t>(1, kSweepBudget / sw_per_block));

  size_t off = 0;
  auto take = [&](size_t b) {
    size_t o = off;
    off += (b + 255) & ~size_t(255);
    return o;
  };
  g->scratch_ev_heap_off = take(heap_g_bytes * ev_grid);
  g->heap_fill_bytes = heap_g_bytes * ev_grid;
  g->scratch_ev_join_off = take(join_bytes * ev_grid);
  g->scratch_ev_rf_off = take(rf_lds ? 0 : rf_bytes * ev_grid);
  g->scratch_ev_last_off = take(rf_lds ? 0 : rf_bytes * ev_grid);
  g->scratch_at_off = take(P.at_lds ? 0 : (size_t)2 * G.R * kWave * 4 * P.at_blocks);
  g->scratch_cp_off = take(P.cp_mode == kCpSlotsGlobal ? cp_bytes * P.cp_blocks : 0);
  g->scratch_dist_off = take((size_t)std::max(G.n, 1) * 4);
  g->scratch_gen_off = take((size_t)std::max(G.n, 1) * 4);  // one generated duration column
  g->scratch_dev_off = take((size_t)G.R * 8);                 // the device model of a call
  g->scratch_bytes = off;
  // as many eager sets as the pool budget allows (one at least), and one
  // for calls captured into HIP graphs
  const int n_sets = (int)std::max<size_t>(1, std::min<size_t>(kMaxSets, kPoolBudget / std::max<size_t>(off, 1)));
  g->pool.destroy();
  if (int rc = g->pool.init(off, n_sets, true, fill_set, g)) return rc;
  // the sweep's sets (the kernel initialises its state per tile): fewer
  // blocks when the memory is not there
  for (;;) {
    P.sw_blocks = (int32_t)sw_blocks;
    g->scratch_sw_val_off = 0;
    g->scratch_sw_res_off = sw_val_blk * sw_blocks;
    g->sweep_pool.destroy();
    const int rc = g->sweep_pool.init(sw_per_block * sw_blocks, 1, true, nullptr, nullptr);
    if (rc != SIM_E_NOMEM || sw_blocks <= 1) {
      if (rc) return rc;
      break;
    }
    (void)hipGetLastError();  // clear the failed allocation's error
    sw_blocks = std::max<size_t>(1, sw_blocks / 2);
  }
  if (getenv("MLSIM_VERBOSE"))  // diagnostics only
    fprintf(stderr,
            "[mlsim] n=%d R=%d J=%d (barriers %d) heap_cap=%d (stride %d, lds end %d) cp_slots=%d (mode %d) "
            "ev_blocks=%d cp_blocks=%d sw_blocks=%d ev_lds=%zu scratch=%zu MB x %d sets\n",
            G.n, G.R, G.J, g->n_barriers, G.heap_cap, P.ev_heap_stride, P.ev_heap_le, G.cp_slots, P.cp_mode,
            P.ev_blocks, P.cp_blocks, P.sw_blocks, P.ev_lds_bytes, off >> 20, n_sets);
  return SIM_OK;
}

namespace {
// Per-block scratch of the event kernel outside a graph's scratch sets: the
// heap's global levels, join state and (when not in LDS) resource times, each
// indexed by block, for at most max_blocks blocks.
struct EvScratch {
  uint64_t *heap;
  int2 *join;
  uint32_t *rf;
  int64_t max_blocks;
};

int launch_event_impl(const sim_graph *g, char *base, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                      const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                      int64_t ld_fin, int32_t *status, int32_t *prev, hipStream_t stream,
                      const DurGen *gen = nullptr, const int32_t *dev = nullptr, bool has_gap = false,
                      bool has_delay = false, const EvScratch *ext = nullptr) {
  const ScratchPlan &P = g->plan;
  EvArgs a{n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin, status,
           ext ? ext->heap : (uint64_t *)(base + g->scratch_ev_heap_off), P.ev_heap_stride, P.ev_heap_le,
           ext ? ext->join : (int2 *)(base + g->scratch_ev_join_off),
           ext ? ext->rf : (uint32_t *)(base + g->scratch_ev_rf_off),
           prev, ext ? nullptr : (int32_t *)(base + g->scratch_ev_last_off), P.ev_last16, DurGen{}, dev, has_gap,
           has_delay};
  if (gen) a.gen = *gen;
  const int64_t tiles = (n_scen + kWave - 1) / kWave;
  const bool rf_lds = P.rf_lds;
  const dim3 block(kWave);
  // when the last round of tiles would fill less than half the grid, use
  // fewer blocks that each take the same number of tiles (within one)
  // registers for the heap root's children when the chip is full: the
  // variant with the children in LDS would need two or more rounds of tiles
  const int64_t lds_blocks = prev ? P.ev_prev_blocks : gen ? P.ev_gen_blocks : dev ? P.ev_dev_blocks : P.ev_blocks;
  bool reg = P.ev_reg && !place && tiles >= 2 * lds_blocks;
  if (g->var.ev_reg >= 0) reg = P.ev_reg && !place && g->var.ev_reg != 0;
  int64_t blocks = !reg ? lds_blocks
                   : prev ? P.ev_reg_prev_blocks
                   : gen  ? P.ev_reg_gen_blocks
                   : dev  ? P.ev_reg_dev_blocks
                          : P.ev_reg_blocks;
  size_t lds = reg ? (prev ? P.ev_reg_prev_lds_bytes : P.ev_reg_lds_bytes)
                   : (prev ? P.ev_prev_lds_bytes : P.ev_lds_bytes);
  if (!reg && !ext) {  // few tiles: the whole third heap level in LDS
    const int64_t wide = prev ? P.ev_wide_prev_blocks
                         : gen ? P.ev_wide_gen_blocks
                         : dev ? P.ev_wide_dev_blocks
                               : P.ev_wide_blocks;
    if (tiles <= wide) {
      blocks = wide;
      a.heap_le = P.ev_wide_le;
      lds = P.ev_wide_lds_bytes + (prev && rf_lds ? (size_t)g->dg.R * kWave * (P.ev_last16 ? 2 : 4) : 0);
    }
  }
  if (ext) blocks = std::min(blocks, ext->max_blocks);
  const int64_t rounds = (tiles + blocks - 1) / blocks;
  const int64_t tail = tiles - (rounds - 1) * blocks;
  const dim3 grid((unsigned)(2 * tail >= blocks ? std::min<int64_t>(tiles, blocks)
                                                : (tiles + rounds - 1) / rounds));
  const int variant = (reg && !gen && !prev && !dev ? 128 : 0) | (reg ? 64 : 0) | (gen ? 16 : 0) | (prev ? 8 : 0) |
                      (rf_lds ? 4 : 0) | (g->dg.ev_compact ? 2 : 0) | (place ? 1 : 0);
#define EV_CASE(V, A, B, C, D) \
  case V: k_event<A, B, C, D><<<grid, block, lds, stream>>>(g->dg, a); break;
#define EV_GEN_CASE(V, A, B) \
  case V: k_event<A, B, false, false, true><<<grid, block, lds, stream>>>(g->dg, a); break;
#define EV_REG_CASE(V, B, D, E) \
  case V: k_event<true, B, false, D, E, true><<<grid, block, lds, stream>>>(g->dg, a); break;
  switch (variant) {
    // the heap root's children in registers (loaded durations, no device
    // model: the heap's last element read only when a pop needs it)
    case 196: k_event<true, false, false, false, false, true, true><<<grid, block, lds, stream>>>(g->dg, a); break;
    case 198: k_event<true, true, false, false, false, true, true><<<grid, block, lds, stream>>>(g->dg, a); break;
    EV_REG_CASE(68, false, false, false)
    EV_REG_CASE(70, true, false, false)
    EV_REG_CASE(76, false, true, false)
    EV_REG_CASE(78, true, true, false)
    EV_REG_CASE(84, false, false, true)
    EV_REG_CASE(86, true, false, true)
    EV_GEN_CASE(16, false, false)
    EV_GEN_CASE(18, false, true)
    EV_GEN_CASE(20, true, false)
    EV_GEN_CASE(22, true, true)
    EV_CASE(0, false, false, false, false)
    EV_CASE(1, false, false, true, false)
    EV_CASE(2, false, true, false, false)
    EV_CASE(3, false, true, true, false)
    EV_CASE(4, true, false, false, false)
    EV_CASE(5, true, false, true, false)
    EV_CASE(6, true, true, false, false)
    EV_CASE(7, true, true, true, false)
    EV_CASE(8, false, false, false, true)
    EV_CASE(9, false, false, true, true)
    EV_CASE(10, false, true, false, true)
    EV_CASE(11, false, true, true, true)
    EV_CASE(12, true, false, false, true)
    EV_CASE(13, true, false, true, true)
    EV_CASE(14, true, true, false, true)
    default: k_event<true, true, true, true><<<grid, block, lds, stream>>>(g->dg, a); break;
  }
#undef EV_CASE
#undef EV_GEN_CASE
#undef EV_REG_CASE
  return hipGetLastError() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

// Generated durations written out: dur[v * ld + s] for every op and scenario
// (one thread per scenario column, blocks striding over ops; each store row
// of a block is 1 KB contiguous).
__global__ __launch_bounds__(256) void k_generate(DurGen gen, int64_t n_scen, int32_t *dur, int64_t ld) {
  const int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (s >= n_scen) return;
  const int64_t S = gen.scen0 + s;
  const int32_t *brow = gen_knob_row(gen, S);
  const uint32_t s_lo = (uint32_t)S, s_hi = (uint32_t)((uint64_t)S >> 32);
  for (int32_t v = blockIdx.y; v < gen.n_ops; v += gridDim.y)
    dur[(int64_t)v * ld + s] = gen_duration(brow[v], s_lo, s_hi, (uint32_t)v, gen.key0, gen.key1, gen.noise);
}
}  // namespace

// Up to kPutWords values passed by value (kernel arguments are captured at
// launch, so the caller's host array may change as soon as the launch
// returns) written to device memory in stream order.
constexpr int kPutWords = 256;
struct PutWords {
  int32_t v[kPutWords];
};
__global__ __launch_bounds__(kPutWords) void k_put_words(int32_t *dst, PutWords w, int count) {
  const int i = threadIdx.x;
  if (i < count) dst[i] = w.v[i];
}

// dst[r * ld + i] = 0 for r < rows, i < count (a kernel rather than a memset,
// so a caller may capture the call in a graph)
__global__ __launch_bounds__(256) void k_zero2d(int32_t *dst, int64_t count, int64_t ld) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < count) dst[(int64_t)blockIdx.y * ld + i] = 0;
}

int launch_zero(int32_t *dst, int64_t count, int64_t ld, int32_t rows, hipStream_t stream) {
  if (!dst || count <= 0 || rows <= 0) return SIM_OK;
  const int64_t xb = (count + 255) / 256;
  for (int32_t r0 = 0; r0 < rows; r0 += 65535) {  // grid y limit
    const int32_t ry = std::min(65535, rows - r0);
    k_zero2d<<<dim3((unsigned)xb, (unsigned)ry), dim3(256), 0, stream>>>(dst + (int64_t)r0 * ld, count, ld);
    if (hipGetLastError() != hipSuccess) return SIM_E_HIP;
  }
  return SIM_OK;
}

int launch_put_words(int32_t *dst, const int32_t *src, int32_t count, hipStream_t stream) {
  for (int32_t k = 0; k < count; k += kPutWords) {
    PutWords w;
    const int32_t m = std::min(kPutWords, count - k);
    memcpy(w.v, src + k, (size_t)m * 4);
    k_put_words<<<1, kPutWords, 0, stream>>>(dst + k, w, m);
    if (hipGetLastError() != hipSuccess) return SIM_E_HIP;
  }
  return SIM_OK;
}

int launch_generate(const DurGen &gen, int64_t n_scen, int32_t *dur, int64_t ld, hipStream_t stream) {
  const int64_t xb = (n_scen + 255) / 256;
  // enough blocks to fill the chip several times over, each op row once
  const int64_t yb = std::min<int64_t>(gen.n_ops, std::max<int64_t>(1, 8192 / xb));
  k_generate<<<dim3((unsigned)xb, (unsigned)yb), dim3(256), 0, stream>>>(gen, n_scen, dur, ld);
  return hipGetLastError() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

int launch_event_dev(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                     const uint16_t *place, int64_t ld_place, const int32_t *dev, bool has_gap,
                     bool has_delay, int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                     hipStream_t stream) {
  return launch_event_impl(g, scr, n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin, status,
                           nullptr, stream, nullptr, dev, has_gap, has_delay);
}

int launch_event_gen(const sim_graph *g, char *scr, int64_t n_scen, const DurGen &gen, int32_t *makespan,
                     int32_t *finish, int64_t ld_fin, int32_t *status, hipStream_t stream) {
  return launch_event_impl(g, scr, n_scen, nullptr, 0, nullptr, 0, makespan, finish, ld_fin, status, nullptr,
                           stream, &gen);
}

int launch_event(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                 const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                 int64_t ld_fin, int32_t *status, hipStream_t stream) {
  return launch_event_impl(g, scr, n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin,
                           status, nullptr, stream);
}

int launch_event_prev(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                      const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                      int32_t *prev, int64_t ld_op, int32_t *status, hipStream_t stream) {
  return launch_event_impl(g, scr, n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_op,
                           status, prev, stream);
}

// Scratch of the replay variant that allocates nothing
// (sim_run_batch_noalloc): one array per GPU in the code object's static
// device memory, held by each GPU the library runs on until the process
// ends.  In host code `scratch` is a stand-in for the symbol, not a device
// address: every host use goes through the address hipGetSymbolAddress
// returned for the device (noalloc_setup), never through the name.
constexpr size_t kNoAllocBytes = (size_t)SIM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kNoAllocBytes];

namespace {
std::mutex g_noalloc_mu;
std::vector<char *> g_noalloc_ptr;  // per device: the array's address, null until looked up

// p[i] = v for i < n (a kernel rather than a memset, so the call can be
// captured in a graph)
__global__ __launch_bounds__(256) void k_fill_words(uint32_t *p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = v;
}

int fill_words(uint32_t *p, int64_t n, uint32_t v, hipStream_t stream) {
  if (n <= 0) return SIM_OK;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  k_fill_words<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(p, n, v);
  return hipGetLastError() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

size_t round256(size_t b) { return (b + 255) & ~size_t(255); }
}  // namespace

int noalloc_setup(int device) {
  std::lock_guard<std::mutex> lk(g_noalloc_mu);
  if (device < 0) return SIM_E_HIP;
  if ((size_t)device >= g_noalloc_ptr.size()) g_noalloc_ptr.resize((size_t)device + 1, nullptr);
  if (g_noalloc_ptr[device]) return SIM_OK;
  void *p = nullptr;  // with `device` current (the caller's)
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SIM_E_HIP;
  g_noalloc_ptr[device] = (char *)p;
  return SIM_OK;
}

int launch_event_noalloc(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                         const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                         int64_t ld_fin, int32_t *status, hipStream_t stream) {
  char *base = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_noalloc_mu);
    if ((size_t)g->device < g_noalloc_ptr.size()) base = g_noalloc_ptr[g->device];
  }
  if (!base) return SIM_E_HIP;
  const ScratchPlan &P = g->plan;
  const DevGraph &G = g->dg;
  // one block's region: heap levels in global memory, join state, resource
  // times when they are not in LDS
  const size_t heap_b = (size_t)P.ev_heap_stride * kWave * 8, join_b = (size_t)G.J * kWave * 8;
  const size_t rf_b = P.rf_lds ? 0 : (size_t)G.R * kWave * 4;
  const size_t per_block = round256(heap_b) + round256(join_b) + round256(rf_b);
  if (per_block > kNoAllocBytes) return SIM_E_LIMIT;
  const int64_t cap = (int64_t)(kNoAllocBytes / per_block);
  const int64_t tiles = (n_scen + kWave - 1) / kWave;
  const int64_t used = std::min(cap, tiles);  // the grid never exceeds the tiles
  EvScratch ext{(uint64_t *)base, (int2 *)(base + (size_t)cap * round256(heap_b)),
                (uint32_t *)(base + (size_t)cap * (round256(heap_b) + round256(join_b))), cap};
  // the previous call may have used another layout: heap positions start
  // empty (all ones) and join state cleared, for every block this call runs
  if (int rc = fill_words((uint32_t *)ext.heap, (int64_t)(used * round256(heap_b) / 4), 0xffffffffu, stream))
    return rc;
  if (int rc = fill_words((uint32_t *)ext.join, (int64_t)(used * round256(join_b) / 4), 0u, stream)) return rc;
  return launch_event_impl(g, nullptr, n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin, status,
                           nullptr, stream, nullptr, nullptr, false, false, &ext);
}

namespace {

using MpKernel = void (*)(MpTable, MpArgs);

template <int M, int O>
MpKernel mp_kernel_of(bool gen, bool bar) {
  if (gen) return bar ? k_maxplus<M, O, true, true> : k_maxplus<M, O, true, false>;
  return bar ? k_maxplus<M, O, false, true> : k_maxplus<M, O, false, false>;
}

// the sweep instance for a slot placement, what it writes, generated
// durations and whether the table holds barrier records
MpKernel mp_kernel(int mode, int out, bool gen, bool bar) {
  if (mode == kCpSlotsLds) {
    if (out == kMpOutFinish) return mp_kernel_of<kCpSlotsLds, kMpOutFinish>(gen, bar);
    if (out == kMpOutDist) return mp_kernel_of<kCpSlotsLds, kMpOutDist>(gen, bar);
    return mp_kernel_of<kCpSlotsLds, kMpOutNone>(gen, bar);
  }
  if (out == kMpOutFinish) return mp_kernel_of<kCpSlotsGlobal, kMpOutFinish>(gen, bar);
  if (out == kMpOutDist) return mp_kernel_of<kCpSlotsGlobal, kMpOutDist>(gen, bar);
  return mp_kernel_of<kCpSlotsGlobal, kMpOutNone>(gen, bar);
}

}  // namespace

int maxplus_occupancy(int mode, bool fin, size_t lds, int cus, bool gen, bool bar) {
  return occupancy_blocks(mp_kernel(mode, fin ? kMpOutFinish : kMpOutNone, gen, bar), lds, cus);
}

int launch_maxplus(const MpTable &T, int mode, int max_blocks, size_t lds, int64_t n_scen,
                   const int32_t *dur, int64_t ld_dur, int32_t *out, int32_t *status,
                   int32_t *finish, int64_t ld_fin, int32_t *dist_out, int64_t dist_scen,
                   uint32_t *slots_g, hipStream_t stream, const DurGen *gen) {
  MpTable t = T;
  MpArgs a{n_scen, dur, ld_dur, out, status, finish, ld_fin, dist_out, dist_scen, slots_g, DurGen{}};
  if (gen) a.gen = *gen;
  const int64_t tiles = (n_scen + kWave - 1) / kWave;
  const dim3 grid((unsigned)std::min<int64_t>(tiles, max_blocks)), blk(kWave);
  const int out_kind = finish ? kMpOutFinish : dist_out ? kMpOutDist : kMpOutNone;
  void *args[] = {&t, &a};
  if (hipLaunchKernel((const void *)mp_kernel(mode, out_kind, gen != nullptr, T.bar != 0), grid, blk, args, lds,
                      stream) != hipSuccess)
    return SIM_E_HIP;
  return hipGetLastError() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

int launch_cp(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
              int32_t *cp_len, int32_t *dist_out, int64_t dist_scen, hipStream_t stream,
              const DurGen *gen) {
  const ScratchPlan &P = g->plan;
  const MpTable T{g->dg.cp_n, g->dg.cp_slots, g->dg.cp, g->dg.cp_pred, g->dg.cp_n > g->dg.n};
  return launch_maxplus(T, P.cp_mode, gen ? P.cp_gen_blocks : P.cp_blocks, P.cp_lds_bytes, n_scen, dur,
                        ld_dur, cp_len, nullptr, nullptr, 0, dist_out, dist_scen,
                        (uint32_t *)(scr + g->scratch_cp_off), stream, gen);
}

int launch_attr(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                const uint16_t *place, int64_t ld_place, const int32_t *finish, const int32_t *prev,
                int64_t ld_op, const int32_t *status, int32_t *busy, int32_t *chain, int64_t ld_res,
                int32_t *chain_ops, hipStream_t stream) {
  const ScratchPlan &P = g->plan;
  AtArgs a{n_scen, dur, ld_dur, place, ld_place, finish, prev, ld_op, status, busy, chain, ld_res,
           chain_ops, (uint32_t *)(scr + g->scratch_at_off)};
  const int64_t tiles = (n_scen + kWave - 1) / kWave;
  const dim3 grid((unsigned)std::min<int64_t>(tiles, P.at_blocks)), blk(kWave);
  const size_t lds = P.at_lds_bytes;
  if (P.at_lds) {
    if (place)
      k_attr<true, true><<<grid, blk, lds, stream>>>(g->dg, a);
    else
      k_attr<false, true><<<grid, blk, lds, stream>>>(g->dg, a);
  } else {
    if (place)
      k_attr<true, false><<<grid, blk, lds, stream>>>(g->dg, a);
    else
      k_attr<false, false><<<grid, blk, lds, stream>>>(g->dg, a);
  }
  return hipGetLastError() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

int launch_sweep(const sim_graph *g, char *base, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                 const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                 int64_t ld_fin, int32_t *status, hipStream_t stream) {
  const ScratchPlan &P = g->plan;
  SwArgs a{n_scen, dur, ld_dur, place, ld_place, makespan, finish, ld_fin, status,
           (uint32_t *)(base + g->scratch_sw_val_off), (uint32_t *)(base + g->scratch_sw_res_off)};
  const int64_t tiles = (n_scen + kWave - 1) / kWave;
  const unsigned blocks = (unsigned)std::min<int64_t>(tiles, P.sw_blocks);
  const size_t lds = P.sw_lds_bytes;
  if (P.sw_val_lds) {
    if (P.sw_res_lds)
      k_sweep<true, true><<<dim3(blocks), dim3(kWave), lds, stream>>>(g->dg, a);
    else
      k_sweep<true, false><<<dim3(blocks), dim3(kWave), lds, stream>>>(g->dg, a);
  } else {
    if (P.sw_res_lds)
      k_sweep<false, true><<<dim3(blocks), dim3(kWave), lds, stream>>>(g->dg, a);
    else
      k_sweep<false, false><<<dim3(blocks), dim3(kWave), lds, stream>>>(g->dg, a);
  }
  return hipGetLastError() == hipSuccess ? SIM_OK : SIM_E_HIP;
}

}  // namespace mlsim
