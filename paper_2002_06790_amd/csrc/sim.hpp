// Internal declarations shared by the host runtime and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <vector>

#include "mlsim.h"
#include "philox.hpp"

namespace mlsim {

constexpr int kWave = 64;  // CDNA wavefront width: one scenario per lane

// Per compact op (ops are renumbered by (priority, id), so "lower compact id"
// is exactly the paper-order tie rule).  Ids n.. are barrier nodes: a set of
// ops that share one predecessor set (two or more predecessors) waits on one
// barrier instead of each counting the predecessors itself; a barrier has no
// duration or resource.  When it completes it releases its first member
// (lowest compact id); each member then releases the next one, at the same
// ready time, through a sibling entry (join index kJoinSibling).  The ops
// whose only predecessor is one op (a fan) may be chained the same way.

// join index of a successor entry: a join counter, or one of these
constexpr int32_t kJoinNone = -1;     // released at the op's finish time
constexpr int32_t kJoinSibling = -2;  // next barrier member, released at the op's ready time
// compact event records only: no entry, and (minus the count of further
// entries) "entries 1.. are in the successor list"
constexpr int32_t kRecNoSucc = -3;
constexpr int32_t kRecMore = -4;
struct OpRec {
  int32_t orig;   // caller's op id: row of dur / place / finish (-1: barrier)
  int32_t res;    // resource (op_res), -1 for a barrier
  int32_t sbeg;   // successor entries succ[sbeg, sbeg + nsucc)
  int32_t nsucc;
  int32_t w0;     // the first two successor entries, repeated here
  int32_t j0;
  int32_t w1;
  int32_t j1;
};

// Per position of the critical-path sweep order (32 bytes): an op, or a
// barrier node standing for a predecessor set that several ops share.  The table is
// padded with empty records (row 0, no slot, no predecessors) to whole
// batches of kCpBatch plus kCpBatch * kCpAhead more, so a sweep can read
// records and rows ahead without bounds checks.
constexpr int kCpBatch = 16;  // ops per batch of the sweep
constexpr int kCpAhead = 4;   // batches of records read ahead
constexpr int kCpSlotsGlobal = 0, kCpSlotsLds = 1;  // where the sweep's value slots live
constexpr int kMpOutNone = 0, kMpOutFinish = 1, kMpOutDist = 2;  // what else the sweep writes
struct CpRec {
  int32_t orig;   // row of dur; -1 for a barrier node (duration 0, no row of its own)
  int32_t slot;   // slot receiving dist(v) (ops without successors: slot cp_slots - 1)
  int32_t npred;
  int32_t pbeg;   // predecessor slots in cp_pred[pbeg, pbeg + npred) when npred > 4
  int32_t p[4];   // the predecessor slots themselves when npred <= 4, then slot
                  // cp_slots - 2, which always holds 0
};

// Device view of a max-plus sweep table (critical path or static-order
// replay): records in sweep order and the long predecessor lists.
struct MpTable {
  int32_t n;      // records swept (ops and barrier nodes)
  int32_t slots;  // value slots (live values + the zero slot + the sink slot)
  const CpRec *rec;
  const int32_t *pred;
  int32_t bar;    // 1 when some records are barrier nodes
};

// Device view of a compiled graph (plain pointers, passed by value).
struct DevGraph {
  int32_t n, R, J, nsrc;  // n real ops (barriers follow them), J join state slots
  int32_t heap_cap;       // bound on simultaneously ready ops (>= DAG width)
  int32_t cp_slots;       // value slots of the critical-path sweep (live values + 2)
  int32_t max_indeg;
  int32_t cp_n;           // records of the critical-path sweep (ops and its barrier nodes)
  const OpRec *ops;       // [n + barriers + 1]
  const int32_t *succ;    // pairs {successor id, its join index, kJoinNone or kJoinSibling}
  const int32_t *jneed;   // [joins] predecessors a join waits for
  const int32_t *src;     // [nsrc] compact ids of sources
  const CpRec *cp;        // [round_up(n, kCpBatch) + kCpBatch * kCpAhead]
  const int32_t *cp_pred; // predecessor slot lists of the critical-path sweep
  const int32_t *pred_ptr;// [n + 1] compact predecessor CSR (sweep variant)
  const int32_t *pred;    // compact predecessor ids
  const int32_t *topo;    // [n] compact ids by (level, id): each level a contiguous range
  const int32_t *lvl_of;  // [n] level of each compact op (longest path from a source)
  const int32_t *levend;  // [levels] last position of each level in topo
  int32_t n_levels, pad3;
  // node graph over 0..n+nb-1 (ops, then barriers; the sharing replay): a barrier's
  // predecessors are its shared set, a member's only predecessor is its
  // barrier; successor lists are the reverse
  int32_t nb, pad1;
  const int32_t *wp_ptr;  // [n+nb+1]
  const int32_t *wp;
  const int32_t *ws_ptr;  // [n+nb+1]
  const int32_t *ws;
  // attribution: predecessors by caller id, ascending ([n+1] CSR), and the
  // resource of each op by caller id
  const int32_t *ap_ptr;
  const int32_t *ap;
  const int32_t *row_res;
  // event kernel: ready-list key words (low 32 bits of a key) are
  // (compact id << pk_sh) | (resource << pk_jb) | join index of the op's
  // first successor entry (pk_jb bits, all ones: not a join), with
  // pk_sh = resource bits + pk_jb (resource bits only with pk_rkey);
  // records, successor entries and sources hold such words for the ops they
  // release directly, and jinfo[j] = {predecessors needed, word released}
  // per join.  With pk_jn a join entry {x, y} itself holds x = the word
  // released and y = join index | predecessors needed << 16, and the join
  // index is a join state slot, which joins never open together may share
  // (without pk_jn each join has its own).
  const OpRec *ev_ops;     // [n + barriers + 1]
  const int32_t *ev_succ;  // pairs {word or barrier id, join index / kJoinNone / kJoinSibling}
  const int2 *jinfo;       // [J]
  const int32_t *ev_src;   // [nsrc]
  int32_t pk_sh, pk_join, pk_jn, pk_jb, pk_rmask;
  // compact event records (identity rows): 16 bytes per op, entries 0 and 1
  // (see kRecNoSucc, kRecMore); the op's resource comes from its key word
  // with pk_rkey, else from row_res
  int32_t ev_compact, pk_rkey;
  const int4 *ev_rec16;
};

struct ScratchPlan {
  int32_t ev_blocks;    // persistent grid of the event kernel
  int32_t ev_heap_stride;  // global heap entries per lane (lane-major, multiple of 16)
  int32_t ev_heap_le;      // first heap position kept in global memory
  int32_t cp_blocks;
  int32_t cp_mode;      // critical-path slots: kCpSlotsLds or kCpSlotsGlobal
  int32_t sw_blocks;
  int32_t sw_val_lds;   // sweep: per-op state in LDS (1) or global (0)
  int32_t sw_res_lds;   // sweep: per-resource state in LDS (1) or global (0)
  size_t ev_lds_bytes, cp_lds_bytes, sw_lds_bytes;
  // attribution: the event kernel with each op's predecessor on its resource
  // (its last-op table beside the resource times), then the chain kernel
  int32_t ev_prev_blocks, at_blocks, at_lds;
  // generated durations: persistent grids of the event and critical-path kernels
  int32_t ev_gen_blocks, cp_gen_blocks;
  int32_t ev_dev_blocks;  // event kernel with a device model (gaps, delays: their table in LDS)
  // event kernel with the heap root's children in registers: available,
  // persistent grids (plain, generated durations, device model) and LDS per block
  int32_t ev_reg, ev_reg_blocks, ev_reg_gen_blocks, ev_reg_dev_blocks, ev_reg_prev_blocks;
  size_t ev_reg_lds_bytes, ev_reg_prev_lds_bytes;
  size_t ev_prev_lds_bytes, at_lds_bytes;
  int32_t rf_lds;       // event kernel: resource times in LDS (1) or global scratch (0)
  int32_t ev_last16;    // attribution's last-op table in 16-bit rows (every row below 0xffff)
  // event kernel with the heap's whole third level in LDS (heap_le
  // ev_wide_le), for calls whose tiles all fit these grids (plain, generated
  // durations, device model, recording predecessors; 0: not planned) and
  // LDS per block (plus the last-op table when recording predecessors)
  int32_t ev_wide_le, ev_wide_blocks, ev_wide_gen_blocks, ev_wide_dev_blocks, ev_wide_prev_blocks;
  size_t ev_wide_lds_bytes;
};

// Kernel variants a graph's launch plan may be pinned to instead of the
// library's choice (every variant computes the same results; the testing
// entry point sim_testing_replan sets these so each one can be checked).
struct Variant {
  int32_t ev_lds_groups = -1;  // heap groups of the root's grandchildren in LDS (0..8), -1: auto
  int32_t ev_blocks_cap = 0;   // cap on the event kernel's persistent grid, 0: none
  int32_t ev_reg = -1;         // heap root's children in registers (0/1), -1: auto
  int32_t cp_global = 0;       // max-plus value slots in global scratch (1) even when LDS holds them
  int32_t rf_global = 0;       // resource times in global scratch (1) even when LDS holds them
  int32_t share_key_id = 0;    // sharing replay: ready-op key words without the resource (1)
};

// A few copies ("sets") of one scratch layout.  Every call takes one set for
// its launches and records an event after them; the next call that takes
// the set first makes its stream wait for that event, so two calls never use
// one set at the same time, whichever streams they run on.  A call prefers
// a set last used on its own stream, then an idle set, then the least
// recently used one.  Calls being captured into a HIP graph use the capture
// set (or set 0 when there is none) without events: such calls cannot wait
// for or record events outside their graph.
struct ScratchPool {
  struct Set {
    char *base = nullptr;
    hipEvent_t done = nullptr;
    hipStream_t last = nullptr;
    bool used = false;
    uint64_t tick = 0;
  };
  std::vector<Set> sets;
  Set capture;  // base == nullptr: captured calls use sets[0]
  size_t bytes = 0;
  uint64_t clock = 0;
  std::mutex mu;
  // allocate n copies of `bytes` (plus the capture copy); init(base) fills
  // one copy's initial contents (stream-ordered on the null stream)
  int init(size_t bytes, int n, bool with_capture, int (*fill)(void *ctx, char *base), void *ctx);
  void destroy();
};

// The set a call uses, held from its first launch until the event after its
// last launch is recorded (the pool's lock is held as long).
class Lease {
 public:
  Lease(ScratchPool &pool, hipStream_t stream);
  ~Lease();
  char *base() const { return set_ ? set_->base : nullptr; }
  int rc() const { return rc_; }
  Lease(const Lease &) = delete;
  Lease &operator=(const Lease &) = delete;

 private:
  ScratchPool &pool_;
  std::unique_lock<std::mutex> lock_;
  ScratchPool::Set *set_ = nullptr;
  hipStream_t stream_;
  bool capturing_ = false;
  int rc_ = 0;
};

}  // namespace mlsim

struct sim_graph {
  int32_t n_ops, n_res;
  int64_t n_edges;  // after dedupe + transitive reduction
  int32_t n_joins, n_levels, n_barriers;
  int32_t row_identity;  // compact id == caller id for every op (no priorities given)
  int device;
  mlsim::DevGraph dg;
  mlsim::ScratchPlan plan;
  mlsim::Variant var;
  void *dev_mem;          // one allocation holding every graph array
  // scratch sets of the event, critical-path and attribution kernels (one
  // layout, offsets below), of the sweep variant (its per-op and
  // per-resource state, offsets below within its own sets) and of the
  // bandwidth-sharing replay; sized here at creation, never allocated by a
  // call
  mutable mlsim::ScratchPool pool, sweep_pool, share_pool;
  size_t scratch_ev_heap_off, scratch_ev_join_off, scratch_ev_rf_off, scratch_cp_off;
  size_t scratch_sw_val_off, scratch_sw_res_off, scratch_dist_off;
  size_t scratch_ev_last_off, scratch_at_off, scratch_gen_off, scratch_dev_off;
  size_t heap_fill_bytes;  // leading bytes of a set that start as all ones (global heap levels)
  // host copies: critical-path recovery (compact predecessor CSR and the
  // caller id of each compact id) and static-order compilation (resource of
  // each op by caller id)
  std::vector<int32_t> h_orig_of, h_pred_ptr, h_pred, h_res;
  size_t scratch_bytes;
  // bandwidth-sharing replay: a set holds the resource flags of the current
  // call, the graph tables below (constant), then the per-block regions of
  // its persistent grid
  int64_t share_head = 0, share_region = 0;  // bytes of flags and tables; of block regions
  int32_t share_slots = 0;                    // nodes with two or more predecessors
  int32_t share_kres = 0, share_rb = 0;       // ready-op key words hold the resource (rb bits)
  std::vector<char> share_tables;             // host copy of the tables (after the flags)
  int64_t share_o_np = 0, share_o_rec = 0, share_o_sent = 0, share_o_mword = 0, share_o_srcw = 0;
};

namespace mlsim {
// bandwidth sharing (share.hip): service units per ns, most active ops per
// resource, persistent grid limits
constexpr uint64_t kShareUnit = SIM_SHARE_UNIT;
constexpr int kShareMax = SIM_SHARE_MAX;
constexpr int64_t kShareBlocksMax = 2048;
constexpr int64_t kShareScratchBudget = (int64_t)8 << 30;
// sizes the sharing replay's scratch and allocates its set (at creation)
int plan_share(sim_graph *g);
int launch_share(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                 const int32_t *share_words, int32_t *makespan, int32_t *finish, int64_t ld_fin,
                 int32_t *status, hipStream_t stream);
// launchers (kernels.hip); scr is the base of the scratch set the call holds
int launch_event(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                 const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                 int64_t ld_fin, int32_t *status, hipStream_t stream);
int launch_sweep(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                 const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                 int64_t ld_fin, int32_t *status, hipStream_t stream);
int launch_cp(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
              int32_t *cp_len, int32_t *dist_out, int64_t dist_scen, hipStream_t stream,
              const DurGen *gen = nullptr);
// generation parameters of a call, checked (SIM_OK or SIM_E_INVAL)
int make_gen(int32_t n_ops, int64_t n_scen, const int32_t *base, int32_t n_knobs, int64_t knob_block,
             uint32_t noise, uint64_t seed, int64_t scen0, DurGen &gen);
// zero rows x count int32 entries (row stride ld) in stream order
int launch_zero(int32_t *dst, int64_t count, int64_t ld, int32_t rows, hipStream_t stream);
// host values copied to device memory in stream order through kernel arguments
int launch_put_words(int32_t *dst, const int32_t *src, int32_t count, hipStream_t stream);
// generated durations: written out, or consumed by the event replay
int launch_generate(const DurGen &gen, int64_t n_scen, int32_t *dur, int64_t ld, hipStream_t stream);
// the event replay with a device model: dev is device memory of 2 n_res
// words (gaps, then output delays); has_gap / has_delay say which apply
int launch_event_dev(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                     const uint16_t *place, int64_t ld_place, const int32_t *dev, bool has_gap,
                     bool has_delay, int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                     hipStream_t stream);
int launch_event_gen(const sim_graph *g, char *scr, int64_t n_scen, const DurGen &gen, int32_t *makespan,
                     int32_t *finish, int64_t ld_fin, int32_t *status, hipStream_t stream);
// attribution: the event replay that also records each op's predecessor on
// its resource, and the busy-time / binding-chain kernel over its outputs
int launch_event_prev(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                      const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                      int32_t *prev, int64_t ld_op, int32_t *status, hipStream_t stream);
int launch_attr(const sim_graph *g, char *scr, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                const uint16_t *place, int64_t ld_place, const int32_t *finish, const int32_t *prev,
                int64_t ld_op, const int32_t *status, int32_t *busy, int32_t *chain, int64_t ld_res,
                int32_t *chain_ops, hipStream_t stream);
// the max-plus sweep on any table: blocks resident per launch for a slot mode
// and LDS size, and the launch itself (finish != null writes finish rows)
int maxplus_occupancy(int mode, bool fin, size_t lds, int cus, bool gen, bool bar);
int launch_maxplus(const MpTable &T, int mode, int max_blocks, size_t lds, int64_t n_scen,
                   const int32_t *dur, int64_t ld_dur, int32_t *out, int32_t *status,
                   int32_t *finish, int64_t ld_fin, int32_t *dist_out, int64_t dist_scen,
                   uint32_t *slots_g, hipStream_t stream, const DurGen *gen = nullptr);
// Records of a max-plus sweep over ops 0..n-1 (duration row of op v:
// row_of[v]) with the given successor and predecessor lists, possibly with
// barrier nodes for shared predecessor sets: the ops in a topological order,
// the value slots, the number of records swept (ops and barriers) and the
// padded records.  extra (empty, or one entry per op): a predecessor of v
// that is left out when predecessor sets are compared, or -1; tie (empty, or
// one key per op): the order preferred among equally good ready ops.  False
// on a cycle.
bool build_maxplus(int32_t n, const std::vector<std::vector<int32_t>> &succ,
                   const std::vector<std::vector<int32_t>> &pred, const std::vector<int32_t> &extra,
                   const std::vector<int64_t> &tie, const std::vector<int32_t> &row_of,
                   std::vector<CpRec> &rec, std::vector<int32_t> &plist, int32_t &slots,
                   std::vector<int32_t> &order, int32_t &n_sweep);
// The static-order replay's sweep table for `order` (a permutation of the
// caller's op ids) over a compiled graph's host view: compact predecessor
// CSR, compact -> caller ids, each caller id's resource.  SIM_E_INVAL for a
// bad order, SIM_E_CYCLE when the order contradicts the DAG.
int static_table(int32_t n, const std::vector<int32_t> &orig_of, const std::vector<int32_t> &pred_ptr,
                 const std::vector<int32_t> &pred_c, const std::vector<int32_t> &res, const int32_t *order,
                 std::vector<CpRec> &rec, std::vector<int32_t> &plist, int32_t &slots, int32_t &n_sweep);
// the replay variant that allocates nothing: the address of the static
// scratch array on the current device, looked up once per device (at graph
// creation), and the launch on it
int noalloc_setup(int device);
int launch_event_noalloc(const sim_graph *g, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                         const uint16_t *place, int64_t ld_place, int32_t *makespan, int32_t *finish,
                         int64_t ld_fin, int32_t *status, hipStream_t stream);
// sizing of persistent grids and LDS, decided once per graph (and again by
// sim_testing_replan), and the allocation of the graph's scratch sets
int plan_scratch(sim_graph *g);
}  // namespace mlsim
