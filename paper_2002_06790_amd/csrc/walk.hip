// gfx950 kernels of the lockstep walk: the replay of many scenarios along one
// shared op order, exact per scenario.
//
// Why it is exact.  With durations >= 1 the schedule of a scenario is unique:
// the only per-resource orders that are sorted by the (ready time, priority,
// id) keys they produce, with start = max(ready, previous finish on the
// resource), are the discrete-event result of the paper's replay loop (Sec.
// 2, "Dataflow based simulation").  So a lane may commit ops in any order that
// respects the graph, as long as every resource receives its ops in strictly
// increasing key order; a lane that ever commits an op with a key not above
// the last key on its resource is flagged, and the exact event kernel replays
// it afterwards.
//
// How it is fast.  Scenarios of one batch are usually close to each other
// (profiled durations vary by about 1 %, Sec. 3), so most of them order each
// resource the same way.  k_pilot replays one scenario per group of tiles with
// the event loop and records its pop order; k_walk then walks that order with
// all 64 lanes of a wave in lockstep, so every duration and finish row is one
// coalesced 256-byte access.  Where a lane's keys order two ops of a resource
// differently from the pilot, the lane commits the later op early ("pulls it
// forward") when its ready time is already known; this covers the common case
// of an op whose inputs arrived a little earlier in that scenario.
#include <algorithm>
#include <cstdio>
#include <cstdlib>

#include "regarr.hpp"
#include "sim.hpp"

extern "C" __device__ uint32_t __ockl_wfred_min_u32(uint32_t);

namespace mlsim {

namespace {

constexpr uint32_t kI32Max = 0x7fffffffu;

template <class T>
using cptr = const __attribute__((address_space(4))) T *;
template <class T>
__device__ __forceinline__ cptr<T> as_const(const T *p) {
  return (cptr<T>)p;
}

__device__ __forceinline__ int32_t uni(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ uint32_t uni(uint32_t x) { return (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)x); }

__device__ __forceinline__ uint64_t make_key(uint32_t ready, int32_t c) {
  return ((uint64_t)ready << 32) | (uint32_t)c;
}

__device__ __forceinline__ OpRec load_op(cptr<OpRec> p, int k) {
  OpRec r;
  r.orig = p[k].orig;
  r.res = p[k].res;
  r.sbeg = p[k].sbeg;
  r.nsucc = p[k].nsucc;
  r.w0 = p[k].w0;
  r.j0 = p[k].j0;
  r.w1 = p[k].w1;
  r.j1 = p[k].j1;
  return r;
}

}  // namespace

// ---------------------------------------------------------------------------
// k_pilot: one wave per group.
//
// Phase A replays the group's first scenario exactly like k_event (same keys,
// joins, barriers and chained barrier members), with every piece of state in
// LDS: the scenario's durations (gathered once), the resource times, the join
// counters and the ready list, kept as an unsorted array whose minimum the
// wave finds with two 32-bit wave reductions.  Its pop order is the walk
// order of the group.
//
// Phase B compiles the walk program.  Positions: op v = T[k] sits at k; a
// barrier is evaluated right after its last predecessor.  A value (finish
// time of an op, or a barrier's maximum) lives in a slot from its position to
// the position of its last consumer; slots are assigned greedily.  Per
// position the program lists the op's row, resource, compact id, output slot,
// predecessor slots, the barriers evaluated after it, the next kCand ops on
// the same resource (the pull-forward candidates) and the compact id of the
// previous op on the resource.  Per position it also describes the op for its
// use as a candidate: the largest position among its predecessors other than
// a same-resource "chain" predecessor, their slots, and the chain predecessor
// (the predecessor with the largest position, when it runs on the same
// resource).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kWave) void k_pilot(DevGraph G, WalkArgs a) {
  extern __shared__ uint32_t lds[];
  const int lane = threadIdx.x;
  const int n = G.n, N = G.n + G.nb, R = G.R, J = G.J;
  const cptr<OpRec> ops = as_const(G.ops);
  const cptr<int32_t> succ = as_const(G.succ);
  const cptr<int32_t> jneed = as_const(G.jneed);
  const cptr<int32_t> wpp = as_const(G.wp_ptr);
  const cptr<int32_t> wp = as_const(G.wp);

  // LDS carve-up (words)
  uint32_t *dcol = lds;                        // [n]  phase A durations; phase B: next position on the resource
  int32_t *posl = (int32_t *)(dcol + n);       // [N]
  int32_t *lastl = posl + N;                   // [N]
  int32_t *slotl = lastl + N;                  // [N]
  int32_t *Tl = slotl + N;                     // [n]
  uint32_t *rf = (uint32_t *)(Tl + n);         // [R]  phase B: last position per resource
  int2 *jst = (int2 *)(rf + R);                // [J]
  uint64_t *rs = (uint64_t *)(jst + J);        // [cap] ready list; phase B: slot expiry
  int32_t *bord = (int32_t *)(rs + a.rs_cap);  // [nb] barriers by evaluation position

  if (blockIdx.x == 0 && lane == 0) *a.retry_count = 0;  // k_walk appends after this kernel
  for (int g = blockIdx.x; g < a.n_groups; g += gridDim.x) {
    int32_t *gb = a.groups + (size_t)g * a.group_words;
    WalkHdr *hdr = (WalkHdr *)gb;
    int32_t *prog = gb + kHdrWords;
    int32_t *pslot = prog + (size_t)n * kProgWords;
    const int64_t s0 = (int64_t)g * a.tiles_per_group * kWave;  // pilot scenario
    bool ok = true;

    // ---- phase A: exact replay of scenario s0 ----
    for (int c = lane; c < n; c += kWave) {
      int32_t d = a.dur[(int64_t)G.ops[c].orig * a.ld_dur + s0];
      dcol[c] = d < 1 ? 1u : (uint32_t)d;
    }
    for (int r = lane; r < R; r += kWave) rf[r] = 0;
    for (int j = lane; j < J; j += kWave) jst[j] = make_int2(0, 0);
    int cnt = G.nsrc;
    if (cnt > a.rs_cap) ok = false;
    if (ok)
      for (int k = lane; k < G.nsrc; k += kWave) rs[k] = make_key(0, G.src[k]);
    __syncthreads();
    for (int k = 0; k < n && ok; ++k) {
      if (cnt <= 0) {  // cannot happen for a DAG; keeps every index in range
        ok = false;
        break;
      }
      uint64_t best = ~0ull;
      int bi = -1;
      for (int i = lane; i < cnt; i += kWave) {
        const uint64_t x = rs[i];
        if (x < best) {
          best = x;
          bi = i;
        }
      }
      const uint32_t mr = __ockl_wfred_min_u32((uint32_t)(best >> 32));
      const uint32_t mc = __ockl_wfred_min_u32((uint32_t)(best >> 32) == mr ? (uint32_t)best : ~0u);
      const uint64_t win = __ballot(bi >= 0 && (uint32_t)(best >> 32) == mr && (uint32_t)best == mc);
      const int wl = __builtin_ctzll(win);
      const int idx = __builtin_amdgcn_readlane(bi, wl);
      const uint32_t ready = uni(mr);
      const int v = (int)uni(mc);
      const uint64_t lastk = rs[cnt - 1];
      __syncthreads();
      if (lane == 0) {
        rs[idx] = lastk;
        Tl[k] = v;
        posl[v] = k;
      }
      --cnt;
      const OpRec rec = load_op(ops, v);
      const uint32_t d = uni(dcol[v]);
      const uint32_t rfv = uni(rf[rec.res]);
      const uint32_t start = ready > rfv ? ready : rfv;
      uint32_t fin = start + d;
      if (fin > kI32Max) fin = kI32Max;
      if (lane == 0) rf[rec.res] = fin;
      for (int e = 0; e < rec.nsucc; ++e) {
        int w, j;
        if (e == 0) {
          w = rec.w0;
          j = rec.j0;
        } else if (e == 1) {
          w = rec.w1;
          j = rec.j1;
        } else {
          w = succ[2 * (rec.sbeg + e)];
          j = succ[2 * (rec.sbeg + e) + 1];
        }
        uint32_t t;
        if (j == kJoinNone) {
          t = fin;
        } else if (j == kJoinSibling) {
          t = ready;
        } else {
          int2 js = jst[j];
          js.x = uni(js.x) + 1;
          js.y = (uint32_t)uni(js.y) > fin ? uni(js.y) : (int)fin;
          const bool done = js.x >= jneed[j];
          __syncthreads();
          if (lane == 0) jst[j] = js;
          if (!done) continue;
          t = (uint32_t)js.y;
          if (w >= n) w = ops[w].w0;  // a barrier releases its first member
        }
        if (cnt >= a.rs_cap) {
          ok = false;
          break;
        }
        if (lane == 0) rs[cnt] = make_key(t, w);
        ++cnt;
      }
      __syncthreads();
    }
    if (cnt != 0) ok = false;  // every op popped exactly once (a DAG always drains)
    if (!ok) {
      if (lane == 0) {
        hdr->valid = 0;
        hdr->slots = 0;
      }
      continue;
    }

    // ---- phase B: compile the walk program ----
    // barrier evaluation positions; consumers' positions give each value's last use
    for (int b = n + lane; b < N; b += kWave) {
      int m = -1;
      for (int e = wpp[b]; e < wpp[b + 1]; ++e) m = max(m, posl[wp[e]]);
      posl[b] = m;
    }
    for (int x = lane; x < N; x += kWave) lastl[x] = -1;
    __syncthreads();
    for (int y = lane; y < N; y += kWave) {
      const int cp = posl[y];
      for (int e = wpp[y]; e < wpp[y + 1]; ++e) atomicMax(&lastl[wp[e]], cp);
    }
    // barriers sorted by (evaluation position, id)
    for (int b = n + lane; b < N; b += kWave) {
      const int pb = posl[b];
      int rank = 0;
      for (int b2 = n; b2 < N; ++b2) {
        const int p2 = posl[b2];
        rank += (p2 < pb || (p2 == pb && b2 < b)) ? 1 : 0;
      }
      bord[rank] = b;
    }
    // next position of each position's resource (backward scan), reusing dcol
    int32_t *nxt = (int32_t *)dcol;
    int32_t *lastpos = (int32_t *)rf;
    for (int r = lane; r < R; r += kWave) lastpos[r] = n;
    __syncthreads();
    for (int k = n - 1; k >= 0; --k) {
      const int v = uni(Tl[k]);
      const int r = ops[v].res;
      const int nx = uni(lastpos[r]);
      __syncthreads();
      if (lane == 0) {
        nxt[k] = nx;
        lastpos[r] = k;
      }
    }
    // slot assignment and slot lists, position by position
    int32_t *sexp = (int32_t *)rs;  // [kSlotMax] position of a slot's last use (-1: free)
    for (int s = lane; s < kSlotMax; s += kWave) sexp[s] = -1;
    __syncthreads();
    int off = 0, used = 0, bp = 0;
    for (int k = 0; k < n && ok; ++k) {
      const int v = uni(Tl[k]);
      uint64_t fm0 = __ballot(sexp[lane] < k);
      uint64_t fm1 = __ballot(sexp[lane + kWave] < k);
      auto take_slot = [&](int lastuse) -> int {
        int s;
        if (fm0) {
          s = __builtin_ctzll(fm0);
          fm0 &= fm0 - 1;
        } else if (fm1) {
          s = kWave + __builtin_ctzll(fm1);
          fm1 &= fm1 - 1;
        } else {
          return -1;
        }
        if (lane == 0) sexp[s] = lastuse;
        used = max(used, s + 1);
        return s;
      };
      const int lv = uni(lastl[v]);
      int sv = 0xFFFF;
      if (lv >= 0) {
        sv = take_slot(lv);
        if (sv < 0) {
          ok = false;
          break;
        }
      }
      if (lane == 0) slotl[v] = sv == 0xFFFF ? -1 : sv;
      // slot lists of the position: [np | nbar << 16], np predecessor slots,
      // then per barrier [slot, count, count predecessor slots]
      const int pb = wpp[v], np = wpp[v + 1] - pb;
      const int off0 = off;
      uint32_t packed = 0xFFFFFFFFu;
      for (int e = 0; e < np && e < 4; ++e) {
        const uint32_t sl = (uint32_t)uni(slotl[wp[pb + e]]);
        packed = (packed & ~(0xFFu << (8 * e))) | (sl << (8 * e));
      }
      for (int e = lane; e < np; e += kWave) pslot[off + 1 + e] = slotl[wp[pb + e]];
      off += 1 + np;
      int nbk = 0;
      while (bp < G.nb) {
        const int b = uni(bord[bp]);
        if (uni(posl[b]) != k) break;
        ++bp;
        const int sb = take_slot(uni(lastl[b]));
        if (sb < 0) {
          ok = false;
          break;
        }
        if (lane == 0) slotl[b] = sb;
        const int bb = wpp[b], bn = wpp[b + 1] - bb;
        if (lane == 0) {
          pslot[off] = sb;
          pslot[off + 1] = bn;
        }
        for (int e = lane; e < bn; e += kWave) pslot[off + 2 + e] = slotl[wp[bb + e]];
        off += 2 + bn;
        ++nbk;
      }
      if (!ok) break;
      if (used > a.slot_max) {
        ok = false;
        break;
      }
      if (lane == 0) {
        pslot[off0] = np | (nbk << 16);
        const OpRec rec = load_op(ops, v);
        int32_t *pr = prog + (size_t)k * kProgWords;
        const int sink = G.ws_ptr[v + 1] == G.ws_ptr[v] ? 1 : 0;
        pr[0] = rec.orig;
        pr[1] = (rec.res & 0xFFFF) | (sv << 16);
        const int slow = (np <= 4 && nbk == 0) ? 0 : 1;  // slot lists only in pslot
        pr[2] = v | (slow << 30) | (sink << 31);
        pr[3] = slow ? off0 : (int32_t)packed;
      }
      __syncthreads();
    }
    if (!ok || off > a.pslot_cap) {
      if (lane == 0) {
        hdr->valid = 0;
        hdr->slots = 0;
      }
      continue;
    }
    __syncthreads();
    // the row kAhead positions ahead, and the candidates: among the next kCand
    // ops on the resource (within 127 positions), up to kInlineCand whose
    // predecessors all precede the position (at most 4 of them)
    for (int k = lane; k < n; k += kWave) {
      int32_t *pr = prog + (size_t)k * kProgWords;
      pr[4] = G.ops[Tl[min(k + kAhead, n - 1)]].orig;
      int nc = 0;
      uint32_t cw = 0;
      int p = k;
      for (int j = 0; j < kCand && nc < kInlineCand; ++j) {
        p = nxt[p];
        if (p >= n || p - k > 127) break;
        const int u = Tl[p];
        const int b0 = G.wp_ptr[u], b1 = G.wp_ptr[u + 1];
        if (b1 - b0 > 4) continue;
        int gate = -1;
        uint32_t packed = 0xFFFFFFFFu;
        for (int e = b0; e < b1; ++e) {
          const int q = G.wp[e];
          gate = max(gate, posl[q]);
          const uint32_t sh = 8 * (uint32_t)(e - b0);
          packed = (packed & ~(0xFFu << sh)) | ((uint32_t)slotl[q] << sh);
        }
        if (gate >= k) continue;
        const int sink = G.ws_ptr[u + 1] == G.ws_ptr[u] ? 1 : 0;
        cw |= (uint32_t)(p - k) << (8 * (nc + 1));
        pr[6 + 3 * nc] = u | (sink << 31);
        pr[7 + 3 * nc] = G.ops[u].orig;
        pr[8 + 3 * nc] = (int32_t)packed;
        ++nc;
      }
      pr[5] = (int32_t)(cw | (uint32_t)nc);
    }
    __threadfence();
    if (lane == 0) {
      hdr->valid = 1;
      hdr->slots = used;
    }
  }
}

// ---------------------------------------------------------------------------
// k_walk: one wave per tile of 64 scenarios, all lanes at the same program
// position k (op v on resource r, wave-uniform).  Per lane:
//   - ready = max over v's predecessor slots;
//   - before committing v the lane first commits, smallest key first, (a) the
//     sinks it deferred on r with a smaller key and (b) candidates (the next
//     ops on r) whose predecessors the walk has already passed and whose key
//     is smaller ("pulled forward"); when v itself is a sink (no successors)
//     and a candidate comes first, the lane defers v instead;
//   - every commit on r checks that its key is above the last key on r, then
//     start = max(ready, resource time), finish = start + d.
// Per-lane resource state (time, last key) sits in registers indexed by the
// wave-uniform resource; values of ops live in LDS slots ([slot][64]);
// duration rows stream into an LDS ring kAhead positions ahead with direct
// global-to-LDS loads; the program is read through register windows of 64
// positions (one position per lane, read back with readlane).
// ---------------------------------------------------------------------------
template <int C>
__device__ __forceinline__ int32_t comp(int4 x) {
  return C == 0 ? x.x : C == 1 ? x.y : C == 2 ? x.z : x.w;
}

constexpr int kNsBuf = 4;  // pulled-forward ops with successors awaiting their position

// Append the flagged lanes' scenarios to the retry list (one atomic per wave).
__device__ __forceinline__ void append_retry(const WalkArgs &a, bool flag, int64_t s) {
  const uint64_t bm = __ballot(flag);
  if (!bm) return;
  int base = 0;
  if (threadIdx.x == __builtin_ctzll(bm)) base = atomicAdd(a.retry_list + kRetryCap, __popcll(bm));
  base = __builtin_amdgcn_readlane(base, __builtin_ctzll(bm));
  const int off = __builtin_amdgcn_mbcnt_hi((uint32_t)(bm >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bm, 0));
  if (flag && base + off < kRetryCap) a.retry_list[base + off] = (int32_t)s;
}

// FIN: finish times are written; NR: registers for the per-resource state;
// ROW_ID: every op's row equals its compact id.
template <bool FIN, int NR, bool ROW_ID>
__global__ __launch_bounds__(kWave) void k_walk(DevGraph G, WalkArgs a) {
  extern __shared__ uint32_t lds[];
  const int lane = threadIdx.x;
  const int n = G.n;
  uint32_t *slots = lds + lane;                                         // [slot_max][64]
  uint32_t *ring0 = lds + (size_t)a.slot_max * kWave;                   // [kRing][64]
  uint16_t *lastc = (uint16_t *)(ring0 + (size_t)kRing * kWave) + lane; // [R][64] compact id of the last commit
  const int64_t tiles = (a.n_scen + kWave - 1) / kWave;
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const int64_t s = tile * kWave + lane;
    const bool active = s < a.n_scen;
    const int64_t sc = active ? s : a.n_scen - 1;
    const int g = (int)(tile / a.tiles_per_group);
    const int32_t *gb = a.groups + (size_t)g * a.group_words;
    if (!uni(*(const volatile int32_t *)gb)) {
      if (active) a.makespan[s] = kWalkRetry;
      append_retry(a, active, s);
      continue;
    }
    const int4 *prog4 = (const int4 *)(gb + kHdrWords);
    const cptr<int32_t> pslot = as_const(gb + kHdrWords + (size_t)n * kProgWords);
    // program windows: lane i holds the record of position B + i (W0) and
    // B + 64 + i (W1); the walk only reads W0, W1 arrives in the background
    int4 a0, a1, a2, a3, b0, b1, b2, b3;
    auto load_win = [&](int base, int4 &x0, int4 &x1, int4 &x2, int4 &x3) {
      const int p = base + lane;
      if (p < n) {
        x0 = prog4[4 * (size_t)p];
        x1 = prog4[4 * (size_t)p + 1];
        x2 = prog4[4 * (size_t)p + 2];
        x3 = prog4[4 * (size_t)p + 3];
      } else {
        x0 = x1 = x2 = x3 = make_int4(0, 0, 0, 0);
      }
    };
    load_win(0, a0, a1, a2, a3);
    load_win(64, b0, b1, b2, b3);
    int B = 0;
    auto ring_load = [&](int p, int row) {  // request position p's durations (row) into the ring
      if ((unsigned)row >= (unsigned)n) row = 0;  // rows come from the program; keep them in range
      __builtin_amdgcn_global_load_lds((const void *)(a.dur + (int64_t)row * a.ld_dur + sc),
                                       (__attribute__((address_space(3))) void *)(ring0 + (p & (kRing - 1)) * kWave),
                                       4, 0, 0);
    };
    // ring loads of the previous tile (requested past its end, or cut short
    // by an abort) land before this tile's requests reuse their slots
    __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
    for (int p = 0; p < kAhead; ++p) ring_load(p, __builtin_amdgcn_readlane(a0.x, min(p, n - 1)));

    RegArr<NR> rf, lr;  // resource time; ready time of the last commit (-1: none)
    rf.fill(0u);
    lr.fill(~0u);
    for (int r = 0; r < G.R; ++r) lastc[r * kWave] = 0;
    uint64_t done_lo = 0, done_hi = 0;  // pulled-forward positions k .. k + 127 (bit p & 127)
    int ns_pos[kNsBuf];
    uint32_t ns_fin[kNsBuf];
#pragma unroll
    for (int i = 0; i < kNsBuf; ++i) {
      ns_pos[i] = -1;
      ns_fin[i] = 0;
    }
    // deferred sinks: ready, compact id | resource << 16 (resource 0xFFFF: free), duration, row
    uint32_t df_ready[kDefer], df_cr[kDefer], df_d[kDefer], df_row[ROW_ID ? 1 : kDefer];
#pragma unroll
    for (int e = 0; e < kDefer; ++e) {
      df_ready[e] = 0;
      df_cr[e] = 0xFFFF0000u;
      df_d[e] = 0;
      if (!ROW_ID) df_row[e] = 0;
    }
    uint64_t dres = 0;  // resources with deferred sinks
    bool fail = false;
    uint32_t span = 0;
    // Commit an op on the wave-uniform resource r for the lanes with en set.
    // Every lane executes it (uniform control flow keeps the register-indexed
    // arrays in place); lanes without en keep their state.
    auto commit = [&](bool en, int r, uint32_t t, uint32_t cc, int32_t d) -> uint32_t {
      const bool bad_d = d < 1;
      if (bad_d) d = 1;
      const uint32_t lrv = lr.get(r), lcv = lastc[r * kWave], rfv = rf.get(r);
      const bool later = (int)t > (int)lrv || (t == lrv && cc > lcv);
      const uint32_t st = t > rfv ? t : rfv;
      uint32_t f = st + (uint32_t)d;
      const bool ovf = f > kI32Max;
      if (ovf) f = kI32Max;
      if (en && (bad_d || !later || ovf)) fail = true;
      lr.set(r, en ? t : lrv);
      rf.set(r, en ? f : rfv);
      lastc[r * kWave] = (uint16_t)(en ? cc : lcv);
      if (en) span = f > span ? f : span;
      return f;
    };
    auto store_fin = [&](int row, uint32_t f) {
      if (FIN && active && (unsigned)row < (unsigned)n) a.finish[(int64_t)row * a.ld_fin + s] = (int32_t)f;
    };
    auto slots_max = [&](uint32_t packed) -> uint32_t {
      uint32_t m = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t sl = (packed >> (8 * e)) & 0xFFu;
        if (sl != 0xFFu) {
          const uint32_t x = slots[sl * kWave];
          m = x > m ? x : m;
        }
      }
      return m;
    };
    constexpr int KC = kInlineCand;
    // Commit, smallest key first, what must precede key lim on the uniform
    // resource r: deferred sinks on r and valid candidates.  When the op being
    // placed is a sink (sink_v) and a candidate comes first, the lane defers
    // the op instead.
    auto settle = [&](int r, uint64_t lim, bool &busy, bool sink_v, uint32_t v_ready, uint32_t v_c,
                      int32_t v_d, int v_row, int k, bool (&cvalid)[KC], const uint32_t (&cready)[KC],
                      const uint32_t (&cc)[KC], const int (&cpos)[KC], const int (&crow)[KC],
                      const bool (&csink)[KC], bool &deferred) __attribute__((always_inline)) {
      for (int it = 0; it < KC + kDefer + 1; ++it) {
        int choice = -1;  // candidate j, or 100 + e for deferred entry e
        uint64_t best = lim;
        if (busy) {
          if ((dres >> r) & 1) {
#pragma unroll
            for (int e = 0; e < kDefer; ++e) {
              const uint64_t ke = make_key(df_ready[e], (int)(df_cr[e] & 0xFFFFu));
              if ((int)(df_cr[e] >> 16) == r && ke < best) {
                best = ke;
                choice = 100 + e;
              }
            }
          }
#pragma unroll
          for (int j = 0; j < KC; ++j) {
            const uint64_t kj = make_key(cready[j], (int)cc[j]);
            if (cvalid[j] && kj < best) {
              best = kj;
              choice = j;
            }
          }
        }
        if (!__ballot(choice >= 0)) break;
        const bool is_def = choice >= 100, is_cand = choice >= 0 && choice < 100;
        uint32_t t_sel = 0, c_sel = 0, d_def = 0;
        int row_sel = 0, p_sel = 0;
        bool s_sel = false;
        // per-entry selects (a dynamically indexed update would move the list to memory)
        const uint32_t hit = is_def ? 1u << (choice - 100) : 0u;
#pragma unroll
        for (int e = 0; e < kDefer; ++e) {
          const bool h = (hit >> e) & 1u;
          t_sel = h ? df_ready[e] : t_sel;
          c_sel = h ? (df_cr[e] & 0xFFFFu) : c_sel;
          d_def = h ? df_d[e] : d_def;
          if (!ROW_ID) row_sel = h ? (int)df_row[ROW_ID ? 0 : e] : row_sel;
          df_cr[e] = h ? 0xFFFF0000u : df_cr[e];
        }
        if (ROW_ID && is_def) row_sel = (int)c_sel;
#pragma unroll
        for (int j = 0; j < KC; ++j) {
          const bool h = choice == j;
          t_sel = h ? cready[j] : t_sel;
          c_sel = h ? cc[j] : c_sel;
          p_sel = h ? cpos[j] : p_sel;
          row_sel = h ? crow[j] : row_sel;
          s_sel = h ? csink[j] : s_sel;
          cvalid[j] = h ? false : cvalid[j];
        }
        if (sink_v && is_cand) {  // the sink goes after the candidate: defer it
          bool placed = false;
#pragma unroll
          for (int e = 0; e < kDefer; ++e) {
            const bool h = !placed && (df_cr[e] >> 16) == 0xFFFFu;
            df_ready[e] = h ? v_ready : df_ready[e];
            df_cr[e] = h ? (v_c | ((uint32_t)r << 16)) : df_cr[e];
            df_d[e] = h ? (uint32_t)v_d : df_d[e];
            if (!ROW_ID) df_row[ROW_ID ? 0 : e] = h ? (uint32_t)v_row : df_row[ROW_ID ? 0 : e];
            placed |= h;
          }
          if (!placed) fail = true;
          dres |= 1ull << r;
          deferred = true;
          busy = false;
        }
        const bool en = choice >= 0 && !(sink_v && is_cand);
        int32_t dsel = (int32_t)d_def;
        if (is_cand && en) {
          if (p_sel - k <= kAhead - kLat)
            dsel = (int32_t)ring0[(p_sel & (kRing - 1)) * kWave + lane];
          else if ((unsigned)row_sel < (unsigned)n)
            dsel = a.dur[(int64_t)row_sel * a.ld_dur + sc];
          else
            fail = true;
        }
        const uint32_t f = commit(en, r, t_sel, c_sel, dsel);
        if (en) {
          store_fin(row_sel, f);
          if (is_cand) {
            const int cb = p_sel & 127;
            if (cb < 64)
              done_lo |= 1ull << cb;
            else
              done_hi |= 1ull << (cb - 64);
            if (!s_sel) {
              bool placed = false;
#pragma unroll
              for (int i = 0; i < kNsBuf; ++i) {
                const bool h = !placed && ns_pos[i] < 0;
                ns_pos[i] = h ? p_sel : ns_pos[i];
                ns_fin[i] = h ? f : ns_fin[i];
                placed |= h;
              }
              if (!placed) fail = true;
            }
          }
        }
        if (is_def) {
          bool left = false;
#pragma unroll
          for (int e = 0; e < kDefer; ++e) left |= (int)(df_cr[e] >> 16) == r;
          if (!left) dres &= ~(1ull << r);
        }
      }
    };

    constexpr int kVm = FIN ? 2 * kLat : kLat;  // VMEM operations newer than the row needed now
    bool aborted = false;
    for (int k = 0; k < n; ++k) {
      if ((k & 255) == 255 &&
          2 * __popcll(__ballot(active && fail)) > __popcll(__ballot(active))) {
        aborted = true;  // most scenarios of this tile need the event replay anyway
        break;
      }
      if (k - B == 64) {
        B = k;
        a0 = b0;
        a1 = b1;
        a2 = b2;
        a3 = b3;
        load_win(k + 64, b0, b1, b2, b3);
      }
      const int l = k - B;
#define RL(x) __builtin_amdgcn_readlane((x), l)
      int row = RL(a0.x);
      if ((unsigned)row >= (unsigned)n) {  // a damaged program flags the tile instead of faulting
        row = 0;
        fail = true;
      }
      const int w1 = RL(a0.y);
      const int w2 = RL(a0.z);
      const uint32_t w3 = (uint32_t)RL(a0.w);
      ring_load(k + kAhead, RL(a1.x));
      // vmcnt(kVm): the row requested kLat steps ago (and everything older) has arrived
      __builtin_amdgcn_s_waitcnt((kVm & 15) | ((kVm >> 4) << 14) | 0x0f70);
      const uint32_t cw = (uint32_t)RL(a1.y);
      const int r = w1 & 0xFFFF, sv = (int)((uint32_t)w1 >> 16);
      const uint32_t c = (uint32_t)w2 & 0x3fffffffu;
      const bool sink = w2 < 0;
      const bool slow = ((uint32_t)w2 >> 30) & 1u;  // slot lists in pslot: many predecessors or barriers
      const int32_t d = (int32_t)ring0[(k & (kRing - 1)) * kWave + lane];
      // pulled forward earlier?
      const int bit = k & 127;
      bool done_v;
      if (bit < 64) {
        done_v = (done_lo >> bit) & 1;
        done_lo &= ~(1ull << bit);
      } else {
        done_v = (done_hi >> (bit - 64)) & 1;
        done_hi &= ~(1ull << (bit - 64));
      }
      uint32_t fin = 0;
      if (done_v && !sink) {
#pragma unroll
        for (int i = 0; i < kNsBuf; ++i) {
          const bool h = ns_pos[i] == k;
          fin = h ? ns_fin[i] : fin;
          ns_pos[i] = h ? -1 : ns_pos[i];
        }
      }
      uint32_t ready = 0;
      int off = 0, np = 0, nbk = 0;
      if (!slow) {
        ready = slots_max(w3);
      } else {
        off = (int)w3;
        if ((unsigned)off < (unsigned)a.pslot_cap) {
          const int hd = pslot[off];
          np = hd & 0xFFFF;
          nbk = hd >> 16;
        }
        if (off + 1 + np > a.pslot_cap) {
          np = nbk = 0;
          fail = true;
        }
        for (int e = 0; e < np; ++e) {
          const uint32_t x = slots[pslot[off + 1 + e] * kWave];
          ready = x > ready ? x : ready;
        }
      }
      bool busy = !done_v, deferred = false;
      const uint64_t kv = make_key(ready, (int)c);
      const int nc = (int)(cw & 0xFFu);
      bool need = false;
      if (__ballot(busy && ((dres >> r) & 1))) {
        // a deferred sink on r goes first only if it became ready no later than v
        uint32_t dm = ~0u;
#pragma unroll
        for (int e = 0; e < kDefer; ++e)
          if ((int)(df_cr[e] >> 16) == r && df_ready[e] < dm) dm = df_ready[e];
        need = busy && dm <= ready;
      }
      uint32_t cready[KC], cc[KC];
      bool cvalid[KC], csink[KC];
      int cpos[KC], crow[KC];
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        cvalid[j] = false;
        cready[j] = cc[j] = 0;
        cpos[j] = crow[j] = 0;
        csink[j] = false;
      }
      if (nc > 0) {
        const int4 cx[3] = {make_int4(RL(a1.z), RL(a1.w), RL(a2.x), 0), make_int4(RL(a2.y), RL(a2.z), RL(a2.w), 0),
                            make_int4(RL(a3.x), RL(a3.y), RL(a3.z), 0)};
#pragma unroll
        for (int j = 0; j < KC; ++j) {
          if (j >= nc) break;
          const int p = k + (int)((cw >> (8 * (j + 1))) & 0xFFu);
          cpos[j] = p;
          cc[j] = (uint32_t)cx[j].x & 0x7fffffffu;
          csink[j] = cx[j].x < 0;
          crow[j] = cx[j].y;
          const int cb = p & 127;
          const bool taken = (((cb < 64 ? done_lo : done_hi) >> (cb & 63)) & 1) != 0;
          cready[j] = slots_max((uint32_t)cx[j].z);
          cvalid[j] = busy && !taken && make_key(cready[j], (int)cc[j]) < kv;
          need |= cvalid[j];
        }
      }
#undef RL
      if (__ballot(need))
        settle(r, kv, busy, sink, ready, c, d, row, k, cvalid, cready, cc, cpos, crow, csink, deferred);
      {
        const uint32_t f = commit(busy, r, ready, c, d);
        if (busy) fin = f;
      }
      if (sv != 0xFFFF && !deferred) slots[sv * kWave] = fin;
      // one finish store per position: lanes that commit v elsewhere write a dummy word
      if (FIN && active) {
        int32_t *dst = (done_v || deferred) ? a.dummy + lane : a.finish + (int64_t)row * a.ld_fin + s;
        *dst = (int32_t)fin;
      }
      // barriers evaluated after v
      if (nbk) {
        int o = off + 1 + np;
        for (int bq = 0; bq < nbk; ++bq) {
          if (o + 2 > a.pslot_cap) {
            fail = true;
            break;
          }
          const int sb = pslot[o], bn = pslot[o + 1];
          if (o + 2 + bn > a.pslot_cap || (unsigned)sb >= (unsigned)a.slot_max) {
            fail = true;
            break;
          }
          uint32_t m = 0;
          for (int e = 0; e < bn; ++e) {
            const uint32_t x = slots[pslot[o + 2 + e] * kWave];
            m = x > m ? x : m;
          }
          slots[sb * kWave] = m;
          o += 2 + bn;
        }
      }
    }
    if (aborted) fail = true;
    // deferred sinks left at the end: each resource in key order
    uint64_t rem = 0;
    if (!aborted)
    for (int i = 0; i < NR; ++i) rem |= __ballot(((dres >> i) & 1) != 0) ? (1ull << i) : 0;
    {
      bool cvalid[KC];
      uint32_t cready[KC], cc[KC];
      int cpos[KC], crow[KC];
      bool csink[KC];
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        cvalid[j] = false;
        cready[j] = cc[j] = 0;
        cpos[j] = crow[j] = 0;
        csink[j] = false;
      }
      while (rem) {
        const int r = __builtin_ctzll(rem);
        rem &= rem - 1;
        bool busy = true, deferred = false;
        settle(r, ~0ull, busy, false, 0, 0, 0, 0, n, cvalid, cready, cc, cpos, crow, csink, deferred);
      }
    }
#pragma unroll
    for (int i = 0; i < kNsBuf; ++i)
      if (ns_pos[i] >= 0) fail = true;  // cannot happen: every position is visited
    if (active) {
      a.makespan[s] = fail ? kWalkRetry : (int32_t)span;
      if (!fail && a.status) a.status[s] = 0;
    }
    append_retry(a, active && fail, s);
  }
}

}  // namespace mlsim

namespace mlsim {

namespace {
constexpr size_t kWalkLdsBudget = 40 * 1024;     // k_walk: four waves per CU
constexpr size_t kPilotLdsBudget = 160 * 1024;   // k_pilot: one wave per CU
constexpr size_t kWalkScratchBudget = 1ull << 30;
}  // namespace

bool walk_eligible(const sim_graph *g) { return g->plan.wk_ok != 0; }

int plan_walk(sim_graph *g, int cus) {
  const DevGraph &G = g->dg;
  ScratchPlan &P = g->plan;
  P.wk_ok = 0;
  P.wk_groups_max = 0;
  P.wk_group_words = 0;
  const int64_t n = G.n, N = G.n + G.nb, R = G.R, J = G.J;
  if (n == 0 || getenv("MLSIM_NO_WALK")) return SIM_OK;
  // k_walk: resource state in registers (up to kWalkMaxRes resources), value
  // slots and the duration ring in LDS
  if (R > kWalkMaxRes || N >= 65536) return SIM_OK;
  const int64_t fixed = (int64_t)kRing * kWave * 4 + (int64_t)R * kWave * 2;  // ring, last compact ids
  if (fixed + 16 * kWave * 4 > (int64_t)kWalkLdsBudget) return SIM_OK;
  P.wk_slot_max = (int32_t)std::min<int64_t>(kSlotMax, ((int64_t)kWalkLdsBudget - fixed) / (kWave * 4));
  P.wk_walk_lds = (size_t)(fixed + (int64_t)P.wk_slot_max * kWave * 4);
  // k_pilot LDS: durations, positions / last uses / slots, order, resource
  // times, joins, ready list, barrier order
  const int64_t base = 4 * n + 12 * N + 4 * n + 4 * R + 8 * J + 4 * (int64_t)G.nb + 64;
  if (base + 8 * 64 > (int64_t)kPilotLdsBudget) return SIM_OK;
  const int64_t cap_room = ((int64_t)kPilotLdsBudget - base) / 8;
  P.wk_rs_cap = (int32_t)std::max<int64_t>(64, std::min<int64_t>(cap_room, (int64_t)G.heap_cap + 64));
  P.wk_pilot_lds = (size_t)(base + 8 * (int64_t)P.wk_rs_cap);
  // per-group program
  int32_t wp_total = 0;
  if (hipMemcpy(&wp_total, G.wp_ptr + N, 4, hipMemcpyDeviceToHost) != hipSuccess) return SIM_E_HIP;
  P.wk_pslot_cap = wp_total + (int32_t)n + 2 * G.nb;
  int64_t words = kHdrWords + n * kProgWords + P.wk_pslot_cap;
  words = (words + 63) & ~int64_t(63);
  P.wk_group_words = words;
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_walk<true, 48, false>, kWave, P.wk_walk_lds) != hipSuccess)
    return SIM_E_HIP;
  if (per_cu < 1) return SIM_OK;
  P.wk_blocks = per_cu * cus;
  int pilot_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&pilot_cu, k_pilot, kWave, P.wk_pilot_lds) != hipSuccess)
    return SIM_E_HIP;
  if (pilot_cu < 1) return SIM_OK;
  // one group per pilot wave the chip holds at once: every pilot runs in the first round
  int64_t gmax = std::min<int64_t>((int64_t)pilot_cu * cus, (int64_t)kWalkScratchBudget / (words * 4));
  if (const char *e = getenv("MLSIM_WALK_GROUPS")) gmax = std::min<int64_t>(gmax, std::max(1, atoi(e)));
  if (gmax < 1) return SIM_OK;
  P.wk_groups_max = (int32_t)gmax;
  P.wk_ok = 1;
  return SIM_OK;
}

int launch_walk(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                hipStream_t stream) {
  const ScratchPlan &P = g->plan;
  const int64_t tiles = (n_scen + kWave - 1) / kWave;
  int64_t tpg = (tiles + P.wk_groups_max - 1) / P.wk_groups_max;
  if (const char *e = getenv("MLSIM_WALK_TPG")) tpg = std::max<int64_t>(tpg, atoi(e));  // tuning override
  const int64_t n_groups = (tiles + tpg - 1) / tpg;
  WalkArgs a{n_scen, dur, ld_dur, makespan, finish, ld_fin, status,
             (int32_t *)((char *)g->scratch + g->scratch_wk_off), P.wk_group_words, (int32_t)n_groups,
             (int32_t)tpg, P.wk_rs_cap, P.wk_slot_max, P.wk_pslot_cap, 0,
             (int32_t *)((char *)g->scratch + g->scratch_wk_off) + (size_t)P.wk_groups_max * P.wk_group_words,
             (int32_t *)((char *)g->scratch + g->scratch_retry_off),
             (int32_t *)((char *)g->scratch + g->scratch_retry_off) + kRetryCap};
  k_pilot<<<dim3((unsigned)n_groups), dim3(kWave), P.wk_pilot_lds, stream>>>(g->dg, a);
  if (hipGetLastError() != hipSuccess) return SIM_E_HIP;
  const unsigned blocks = (unsigned)std::min<int64_t>(tiles, P.wk_blocks);
  const int nr = g->dg.R <= 32 ? 32 : 48;
  const int variant = (finish ? 1 : 0) | (g->row_identity ? 2 : 0);
  const dim3 grid(blocks), blk(kWave);
  const size_t lds = P.wk_walk_lds;
#define WALK_CASE(NR)                                                              \
  switch (variant) {                                                               \
    case 0: k_walk<false, NR, false><<<grid, blk, lds, stream>>>(g->dg, a); break; \
    case 1: k_walk<true, NR, false><<<grid, blk, lds, stream>>>(g->dg, a); break;  \
    case 2: k_walk<false, NR, true><<<grid, blk, lds, stream>>>(g->dg, a); break;  \
    default: k_walk<true, NR, true><<<grid, blk, lds, stream>>>(g->dg, a); break;  \
  }
  if (nr == 32) {
    WALK_CASE(32)
  } else {
    WALK_CASE(48)
  }
#undef WALK_CASE
  if (hipGetLastError() != hipSuccess) return SIM_E_HIP;
  // diagnostics: leave flagged scenarios at kWalkRetry to count them
  if (getenv("MLSIM_WALK_NO_RETRY")) return SIM_OK;
  return launch_event_retry(g, n_scen, dur, ld_dur, makespan, finish, ld_fin, status, a.retry_list,
                            a.retry_count, kRetryCap, stream);
}

}  // namespace mlsim
