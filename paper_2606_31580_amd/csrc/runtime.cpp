// Host runtime of liblaser: model / KV handles, workspace layout, forward planning and the
// hot-path entry points (decode step, confidence probe, mixed step, prefill).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstddef>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

#include "kernels.hpp"
#include "laser.h"
#include "laser_error.h"
#include "pages.hpp"

using namespace laser;

// ----------------------------------------------------------------------------- errors

static thread_local char g_err[512];

extern "C" laser_status laser_fail(laser_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}
extern "C" void laser_clear_error(void) { g_err[0] = 0; }
extern "C" const char* laser_last_error(void) { return g_err; }
extern "C" int laser_abi_version(void) { return LASER_ABI_VERSION; }

#define HIP_TRY(expr)                                                                       \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return laser_fail(LASER_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// Live handles: lets destroy/use of a stale handle fail cleanly instead of touching freed memory.
static std::mutex g_handles_mu;
static std::unordered_set<const void*> g_handles;
static void handle_add(const void* p) {
  std::lock_guard<std::mutex> lk(g_handles_mu);
  g_handles.insert(p);
}
static bool handle_live(const void* p) {
  std::lock_guard<std::mutex> lk(g_handles_mu);
  return p && g_handles.count(p);
}
static void handle_del(const void* p) {
  std::lock_guard<std::mutex> lk(g_handles_mu);
  g_handles.erase(p);
}

// ----------------------------------------------------------------------------- model

namespace {

struct LayerW {
  const void *attn_norm, *wq, *wk, *wv, *bq, *bk, *bv, *wo, *mlp_norm, *w_gate, *w_up, *w_down;
};

constexpr int kRing = 16;   // pinned host staging slots for plan uploads
constexpr int kMaxGraphs = 16;  // captured forwards kept per model (least recently used evicted)
constexpr int kMaxT = 16;   // trial tokens per probe
#ifndef LASER_ATTN_TARGET_WAVES
#define LASER_ATTN_TARGET_WAVES 2048
#endif
constexpr int kTargetAttnWaves = LASER_ATTN_TARGET_WAVES;  // attention waves a forward aims for
// A wave walks its pages with two in flight, so a long run is a chain of memory round trips:
// past the wave target, more waves of at most 4 pages beat longer runs (batch 8 at 68k
// positions: attention + merge 78 -> 61 us per layer; 2 pages: 68 us, 8 pages: 73 us).
#ifndef LASER_ATTN_MAX_PPS
#define LASER_ATTN_MAX_PPS 4
#endif
constexpr int kMaxPagesPerWave = LASER_ATTN_MAX_PPS;
// Splits of a one-row group that merges inside the attention kernel: its last workgroup reads
// every split's partial (G columns x (hd + 2) floats each), so fewer, longer splits shorten
// that tail; the bound trades it against how many workgroups stream the group's pages.
#ifndef LASER_ATTN_FUSED_SPLITS
#define LASER_ATTN_FUSED_SPLITS 56
#endif
constexpr int kFusedMaxSplits = LASER_ATTN_FUSED_SPLITS;
// The split merge runs in the O-projection's launch (mode 1) when the projection's weights
// take at least this many bytes: their stream has to outlast the merge for the merge to be
// hidden (7B shape, 25.7 MB: attention + O-proj 19.7 against 20.1 us per layer with the merge
// kernel; 1.5B shape, 4.7 MB: 15.9 against 15.2 us).
constexpr size_t kMergeMinOBytes = (size_t)16 << 20;

struct Layout {
  size_t rope, h, q, o, act, kpart, kcnt, mcnt, qpart, sqpart, lm_part, attn_part, attn_ml, attn_cnt, plans, probe_p, tok_buf,
      p_buf, total;
  size_t attn_part_bytes, attn_ml_bytes, attn_cnt_bytes, kcnt_bytes, mcnt_bytes;
};

// Launch signature of a forward.  With the plan in its fixed device slot and the caller's
// buffers inside the plan, these values fix every kernel launch of the forward and all of
// its arguments, so one captured graph serves every forward with the same key.
struct FwdKey {
  int M, n_out, agx, mslots, merge;  // agx: attention work items (grid width)
  int mo;                              // the split merge runs in the O-projection's launch
  uint64_t kv_id;
  // same launches apart from the attention grid width
  bool same_shape(const FwdKey& o) const {
    return M == o.M && n_out == o.n_out && mslots == o.mslots && merge == o.merge && mo == o.mo && kv_id == o.kv_id;
  }
};

struct GraphEntry {
  FwdKey key;
  hipGraphExec_t exec;
  uint64_t last_use;
  hipEvent_t done;  // recorded after every kGraphEventEvery-th launch
  int unrecorded;   // launches since done was last recorded
  hipGraph_t graph;           // the captured graph (its nodes address the exec's nodes)
  hipGraphNode_t fetch;       // the plan copy, the forward's first kernel
  hipKernelNodeParams fetch_params;
};

// Every event recorded on the stream between two forwards leaves the GPU idle for a few
// microseconds (between consecutive graph launches of a 7B decode: 22 us with two event
// records and a token copy, 13 us with one event in eight forwards), so completion events are
// recorded only every kGraphEventEvery-th launch of a graph and every kRingEventEvery-th
// plan staging slot.
constexpr int kGraphEventEvery = 8;
constexpr int kRingEventEvery = 8;
static_assert(kRing % kRingEventEvery == 0 && kRing >= 2 * kRingEventEvery, "whole blocks of staging slots");

// Releases a captured forward after its last launch has finished (known from its event, or
// else by waiting for the device: evictions are rare).
static void release_graph(GraphEntry& g) {
  if (g.unrecorded > 0)
    (void)hipDeviceSynchronize();
  else if (g.done)
    (void)hipEventSynchronize(g.done);
  if (g.done) (void)hipEventDestroy(g.done);
  (void)hipGraphExecDestroy(g.exec);
  if (g.graph) (void)hipGraphDestroy(g.graph);
}

// Spans of one kernel class in a timing session: (end of the kernel launched before the
// class's launch, end of the class's last kernel), as indices into the model's event pool.
struct Timer {
  bool enabled = false;
  std::vector<std::pair<int, int>> spans;
};

constexpr int kMaxTimingEvents = 1 << 16;  // per session; later launches go untimed

}  // namespace

struct laser_model {
  laser_model_desc desc;
  int device = 0;
  int cus = 256;  // compute units of the device (set at creation)
  int es = 4;     // bytes per stored weight element
  int kv_es = 4;  // bytes per KV-cache element
  int kv_fp8 = 0; // KV cache in E4M3
  const void* embed = nullptr;
  const void* lm_head = nullptr;
  const void* final_norm = nullptr;
  std::vector<LayerW> layers;
  bool finalized = false;
  int max_rows = 0;
  char* ws = nullptr;
  Layout lay{};
  Plan* h_plans = nullptr;  // pinned ring
  hipEvent_t ring_ev[kRing] = {};
  bool ring_used[kRing] = {};
  int ring_pos = 0;
  long long ring_turn = 0;               // turns of the staging ring so far
  long long ring_rec_turn[kRing] = {};   // the turn in which ring_ev[slot] was last recorded
  Timer timers[LASER_K_NCLASS];
  std::vector<hipEvent_t> ev_pool;  // fence-free timing events, reused across sessions
  int ev_used = 0;
  int last_stop = -1;  // pool index bound to the most recent launch's end
  bool use_graphs = true;
  int gemm_kernel = 0;  // MFMA-path kernel choice (laser_model_set_gemm_kernel)
  // one-row attention groups merge their splits inside the attention kernel (laser_model_set_attn_merge;
  // off by default: measured slower than the merge kernel at the 7B shape, batch 1)
  int attn_fuse = 0;
  int attn_fuse_max = kFusedMaxSplits;
  // where the split merge of 1-2 row forwards runs (laser_model_set_oproj_merge): 0 the merge
  // kernel, 1 the O-projection's launch when its weights hide the merge, 2 the O-projection's
  // launch always; merge_cum: the value each layer's merge counter reaches once
  // every forward launched so far has run; merge_resync: a forward failed after adding to it,
  // so the counters are cleared before the next one
  int oproj_merge = 1;
  unsigned merge_cum = 0;
  bool merge_resync = false;
  // laser_decode_step_static: this device's address of the static scratch array (resolved at
  // finalize) and a host plan buffer, so that the call allocates nothing
  void* static_scratch = nullptr;
  Plan* static_plan = nullptr;
  // tile-order weight copies for the MFMA path (laser_model_set_tiles)
  struct Tiles {
    const char *qkv, *o, *gu, *down;
  };
  std::vector<Tiles> tiles;
  const char* lm_tile = nullptr;
  bool tiles_on = false;
  hipStream_t cap_stream = nullptr;  // private stream that forwards are captured on
  std::vector<GraphEntry> graphs;
  uint64_t graph_clock = 0;
  long long graph_captures = 0;  // forwards captured into graphs since creation

  template <class T>
  T* wsp(size_t off) const { return (T*)(ws + off); }
};

struct laser_kv {
  const laser_model* m;
  uint64_t id;  // unique over the process (graph keys must not match a later cache at the same address)
  PagePool pool;
  void* kpool;
  void* vpool;
  int32_t* bt;
  std::vector<PageUpdate> pending;  // block-table writes not yet on the device
  laser_kv(const laser_model* mm, int np, int ms, int mpps, void* k, void* v, int32_t* b)
      : m(mm), id(next_id()), pool(np, kPage, ms, mpps), kpool(k), vpool(v), bt(b) {}
  static uint64_t next_id() {
    static std::atomic<uint64_t> n{1};
    return n.fetch_add(1);
  }
};

namespace laser {
LaunchEvents& launch_events() {
  static thread_local LaunchEvents ev;
  return ev;
}
}  // namespace laser

namespace {

static int ceil_div(int a, int b) { return (a + b - 1) / b; }
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Projections of up to this many rows run on the VALU path, larger ones on the matrix cores.
// Measured at the 7B shape: at 2 rows the VALU path is faster (riding-probe latency 13.9 vs
// 14.7 ms); at 4 rows the matrix cores are (batch-4 decode step 3.57 vs 4.17 ms: gate/up
// 47.1 vs 58.5 us, LM head 179 vs 295 us).
#ifndef LASER_VALU_MAX_ROWS
#define LASER_VALU_MAX_ROWS 2
#endif
constexpr int kValuMaxRows = LASER_VALU_MAX_ROWS;
static_assert(kValuMaxRows >= 1 && kValuMaxRows <= 4, "VALU kernels exist for 1-4 rows");
static int gemm_mode(int M) { return M <= kValuMaxRows ? M : 4 + ceil_div(M, 16); }

// Workgroups of a projection with `rows` output rows (SwiGLU: gate + up rows) at rw rows each.
static int proj_groups(int epi, int rows, int rw) {
  return epi == EPI_SWIGLU ? ceil_div(rows / 2, rw / 2) : ceil_div(rows, rw);
}

// Rows per workgroup: 16 on the MFMA path (M > kValuMaxRows).  On the VALU path the candidate that
// puts the fewest rows on the busiest compute unit (workgroups dealt round-robin over
// `cus`), larger groups first on ties; QKV groups must tile the rotary pairs exactly.
static int proj_rw(int epi, int rows, int M, int cus) {
  if (M > kValuMaxRows) return rows_per_group(epi, true);
  static const int kQkv[] = {8, 6}, kResid[] = {8, 7, 6}, kOther[] = {8};
  const int* cand = epi == EPI_QKV ? kQkv : (epi == EPI_RESID ? kResid : kOther);
  const int nc = epi == EPI_QKV ? 2 : (epi == EPI_RESID ? 3 : 1);
  int best = 8;
  long long best_cost = -1;
  for (int c = 0; c < nc; ++c) {
    const int rw = cand[c];
    if (epi == EPI_QKV && rows % rw) continue;
    const long long cost = (long long)ceil_div(proj_groups(epi, rows, rw), cus) * rw;
    if (best_cost < 0 || cost < best_cost) {
      best = rw;
      best_cost = cost;
    }
  }
  return best;
}

// Threads per workgroup and chunks (16 bytes of every row) in flight per thread on the VALU
// path, for bf16 weights.  Rows of at most 256 chunks take one chunk per thread, so no thread
// re-reads a clamped chunk and no wave idles (1.5B shape, K = 1536: QKV 6.0 -> 5.5 us,
// gate/up 13.6 -> 10.6 us, LM head 94.7 -> 75.3 us).  Longer residual rows spread over at
// most one workgroup per compute unit take three chunks per thread and cover the row in
// one pass (1.5B down, K = 8960: 7.9 -> 6.95 us).  Everything else keeps the defaults:
// 256 threads (512 for rows over 2,048 chunks) and two chunks, which measured best at the
// 7B shape.  (The other shapes are built for one and two rows of bf16 weights.)
static bool gemv_short_rows(int K, int es, int M) { return es == 2 && M <= 2 && K / 8 <= 256; }

// Rows per QKV workgroup for short rows: four rather than eight when that keeps at most two
// workgroups per compute unit, so that one workgroup's reduction and epilogue overlap the
// other's loads (1.5B shape: QKV 5.5 -> 5.1 us; the residual projections measured no gain).
static int qkv_short_rw(int rows, int cus, int rw) {
  return rows % 4 == 0 && ceil_div(rows, 4) <= 2 * cus ? 4 : rw;
}

static void gemv_shape(int epi, int K, int es, int M, int n_groups, int cus, GemmArgs& a) {
  a.gv_threads = 0;
  a.gv_u = 0;
  if (es != 2 || M > 2) return;
  const int nch = K / 8;
  if (gemv_short_rows(K, es, M)) {
    a.gv_threads = 64 * ceil_div(nch, 64);
    a.gv_u = 1;
  } else if (epi == EPI_RESID && n_groups <= cus && 64 * ceil_div(nch, 3 * 64) <= kGemvMaxThreads) {
    a.gv_threads = 64 * ceil_div(nch, 3 * 64);
    a.gv_u = 3;
  }
}

static int groups_lm(const laser_model_desc& d, int M) { return ceil_div(d.vocab, M > kValuMaxRows ? 16 : 8); }

// Row groups per MFMA workgroup: two (so each activation fragment serves both) when there
// are still at least two workgroups per compute unit; one for the narrow projections and
// for more than one 16-row activation tile.  (Four groups measured slower: more concurrent
// weight streams per wave.)
// Row groups per workgroup, and K shares per row group, on the MFMA path.  A workgroup reads
// its groups' weights and the activation rows over its K range, so several groups per
// workgroup cut the activation reads per weight byte but also the number of workgroups, and
// splitting K (residual projections only: the others normalise over the whole row) restores
// the workgroups at the price of summing the shares.  The choice minimises the bytes read by
// the busiest compute unit (workgroups are dealt round-robin), the sum counted as
// kKsplitPenalty bytes (kKsplit2LongPenalty for two shares of long rows).  At one 16-row
// tile: two groups for gate/up and the LM head, and for QKV at the 7B and 8B shapes (288 or
// 384 groups: 1.2-1.5 workgroups per CU with one group each); with 2-3 tiles up to four
// groups (gate/up of a 40-row mixed step); at 4 tiles up to two.  The down projection splits
// K from 4 rows at the 7B shape (two groups, two shares) and O-proj where the activation rows
// outweigh the weights (the 40-row mixed step).
// MFMA-path kernel and its shape.  nrw = 0: the K-split kernel with nr row groups per
// workgroup; nrw = 1, 2: the row-wave kernel (4 waves of nrw groups each).  ks: K shares.
struct MfmaShape {
  int nr, ks, nrw;
};
constexpr double kKsplitPenalty = 160e3;
// Two shares summed inside the projection (no reduce kernel) cost one more round trip at the
// end of it, which pays only for long rows: for K >= kKsplitLongK the penalty of two shares is
// kKsplit2LongPenalty.  Measured: the 7B batch-4 down projection (K = 18,944) 29.8 -> 26.5 us
// with two shares; with the same penalty at K = 4,096 the 8B batch-8 O-projection took two
// shares and went from 10.6 to 11.4 us.
constexpr double kKsplit2LongPenalty = 40e3;
constexpr int kKsplitLongK = 8192;
#ifndef LASER_RW_MAX_NRW
#define LASER_RW_MAX_NRW 2
#endif
constexpr int kRwMaxGroups = LASER_RW_MAX_NRW;  // row groups per wave of the row-wave kernel, at most
// gemm_kernel: 0 the choice below, 1 only the K-split kernel, 2 the row-wave kernel wherever
// it applies (its shape by the cost below).  The row-wave kernel reads the activations once
// per 4-8 row groups instead of once per 1-4, but streams each group's weights from one wave
// and has few workgroups; measured, it wins for gate/up over 3-4 activation tiles (52 rows at
// 8B: 69 vs 118 us) and for O-proj / down over 4 tiles (32 vs 38 us), and loses where the
// K-split kernel has many workgroups and few activation rows (QKV, the LM head, one tile).
// So by default it takes gate/up at 3-4 tiles when it fills the CUs with 8 groups per
// workgroup, and O-proj / down at 4 tiles (4 groups per workgroup, 4 K shares).  The cost
// for the K-split kernel is the
// bytes the busiest CU reads: ceil(workgroups / CUs) times a workgroup's weights (its groups'
// 16 K es each) and activations (M K 4), over the K shares, plus a fixed penalty for the
// K-share reduce.
static MfmaShape mfma_shape(int epi, int n_groups, int M, int K, int es, int cus, int gemm_kernel) {
  if (M <= kValuMaxRows || M > 64) return {1, 1, 0};
  const int mt = ceil_div(M, 16);
  if (gemm_kernel == 0 && epi == EPI_SWIGLU && mt >= 3 && K % 8 == 0 && ceil_div(n_groups, 8) >= cus * 7 / 8)
    return {1, 1, 2};
  if (gemm_kernel == 0 && epi == EPI_RESID && mt >= 4 && K % 8 == 0) return {1, kMaxKsplit, 1};
  const double w = 16.0 * K * es, act = 4.0 * M * K;
  auto cost = [&](int groups_per_wg, int ks) {
    const double wgs = (double)ceil_div(ceil_div(n_groups, groups_per_wg) * ks, cus);
    const double pen = ks == 2 && K >= kKsplitLongK ? kKsplit2LongPenalty : kKsplitPenalty;
    return wgs * (groups_per_wg * w + act) / ks + (ks > 1 ? pen : 0.0);
  };
  const int max_ks = epi == EPI_RESID ? kMaxKsplit : 1;
  MfmaShape best{1, 1, 0};
  double best_cost = 1e300;
  if (gemm_kernel != 2 || K % 8 != 0)  // (mode 2 falls back to it where K is not a multiple of 8)
    for (int nr : {1, 2, 4}) {
      if (nr == 4 && (mt < 2 || mt > 3)) continue;
      for (int ks = 1; ks <= max_ks; ks *= 2)
        if (cost(nr, ks) < best_cost) {
          best = {nr, ks, 0};
          best_cost = cost(nr, ks);
        }
    }
  if (gemm_kernel == 2 && K % 8 == 0)
    for (int nrw = 1; nrw <= kRwMaxGroups; ++nrw)
      for (int ks = 1; ks <= max_ks; ks *= 2)
        if (cost(4 * nrw, ks) < best_cost) {
          best = {1, ks, nrw};
          best_cost = cost(4 * nrw, ks);
        }
  return best;
}

// QKV over K slices (launch_qkv_slices): forwards of kQSliceMinRows to 64 rows, bf16 weights
// (tile order when the copy is there).  Each workgroup stages a 512-column slice of K of every
// activation row in LDS and runs 16 row groups over it.  Measured against the K-split kernel,
// which reads all of K of every activation row for each of its one or two row groups: QKV of
// the 8B shape at 56 rows 39.3 us against 19.5 + 6.0 us (slices, then their sum and the
// epilogue), at 40 rows 34.0 against 17.1 + 6.0; the 7B shape at 40 rows 30.8 against 14.4 + 6.7.
// Other slice shapes (256 columns; 12 groups per workgroup over 6 waves) measured slower.
constexpr int kQSliceMinRows = 33;
static bool qkv_slices_fit(const laser_model_desc& d, int max_rows) {
  return d.dtype == LASER_DTYPE_BF16 && max_rows >= kQSliceMinRows && d.d_model % 8 == 0 && d.head_dim % 16 == 0;
}

// K-share arrival counters of the residual projections: one per block of their 16-row groups
// (at most d_model / 16 blocks), kKsCntStride apart.
static size_t ks_cnt_bytes(const laser_model_desc& d) {
  return (size_t)ceil_div(d.d_model, 16) * kKsCntStride * 4;
}

static Layout make_layout(const laser_model_desc& d, int max_rows) {
  Layout L{};
  const int hd = d.head_dim, G = d.n_q_heads / d.n_kv_heads;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  L.rope = take((size_t)d.max_positions * (hd / 2) * sizeof(float2));
  L.h = take((size_t)max_rows * d.d_model * 4);
  L.q = take((size_t)max_rows * d.n_q_heads * hd * 4);
  L.o = take((size_t)max_rows * d.n_q_heads * hd * 4);
  L.act = take((size_t)max_rows * d.d_ffn * 4);
  L.kpart = take((size_t)kMaxKsplit * max_rows * d.d_model * 4);  // K-share partials of O-proj / down
  L.kcnt_bytes = ks_cnt_bytes(d);
  L.kcnt = take(L.kcnt_bytes);  // their arrival counters (zero between kernels)
  L.mcnt_bytes = (size_t)d.n_layers * kMgReplicas * kKsCntStride * 4;
  L.mcnt = take(L.mcnt_bytes);  // merge counters of the O-projection's launch (replicas per layer)
  if (qkv_slices_fit(d, max_rows)) {  // K-slice partials of the QKV projection of wide forwards
    const size_t nsl = ceil_div(d.d_model, kQSliceSteps * 32);
    L.qpart = take(nsl * max_rows * (size_t)(d.n_q_heads + 2 * d.n_kv_heads) * hd * 4);
    L.sqpart = take(nsl * max_rows * 4);
  }
  L.lm_part = take((size_t)groups_lm(d, 1) * kMaxRows * sizeof(LmPart));  // the VALU path has the most groups
  L.attn_part_bytes = (size_t)d.n_kv_heads * kAttnMaxWG * max_rows * G * hd * 4;
  L.attn_ml_bytes = (size_t)d.n_kv_heads * kAttnMaxWG * max_rows * G * 2 * 4;
  L.attn_cnt_bytes = (size_t)d.n_kv_heads * kMaxGroups * kAttnCntStride * 4;
  L.attn_part = take(L.attn_part_bytes);
  L.attn_ml = take(L.attn_ml_bytes);
  L.attn_cnt = take(L.attn_cnt_bytes);  // zero between kernels (fused attention merges re-arm them)
  L.plans = take(sizeof(Plan));  // the one device plan slot every forward reads
  L.probe_p = take((size_t)kMaxRows * kMaxT * 4);
  L.tok_buf = take((size_t)kMaxRows * 4);
  L.p_buf = take((size_t)kMaxRows * 4);
  L.total = off;
  return L;
}

static laser_status check_desc(const laser_model_desc* d) {
  if (!d) return laser_fail(LASER_ERR_INVALID_ARG, "desc is NULL");
  if (d->n_layers < 1 || d->d_model < 64 || d->n_q_heads < 1 || d->n_kv_heads < 1 || d->d_ffn < 8 || d->vocab < 2)
    return laser_fail(LASER_ERR_INVALID_ARG, "non-positive model dimension");
  if (d->head_dim != 64 && d->head_dim != 128) return laser_fail(LASER_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (d->n_q_heads % d->n_kv_heads) return laser_fail(LASER_ERR_UNSUPPORTED, "n_q_heads %% n_kv_heads != 0");
  if (d->n_q_heads / d->n_kv_heads > 16) return laser_fail(LASER_ERR_UNSUPPORTED, "query group size above 16");
  if (d->d_model % 64) return laser_fail(LASER_ERR_UNSUPPORTED, "d_model must be a multiple of 64");
  if (d->d_ffn % 8) return laser_fail(LASER_ERR_UNSUPPORTED, "d_ffn must be a multiple of 8");
  if ((d->n_q_heads * d->head_dim) % 64) return laser_fail(LASER_ERR_UNSUPPORTED, "n_q_heads*head_dim % 64 != 0");
  if (d->dtype != LASER_DTYPE_F32 && d->dtype != LASER_DTYPE_BF16) return laser_fail(LASER_ERR_INVALID_ARG, "bad dtype");
  if (d->kv_dtype != 0 && d->kv_dtype != d->dtype && d->kv_dtype != LASER_DTYPE_FP8_E4M3)
    return laser_fail(LASER_ERR_INVALID_ARG, "bad kv_dtype");
  if (d->kv_dtype == LASER_DTYPE_FP8_E4M3 && d->dtype != LASER_DTYPE_BF16)
    return laser_fail(LASER_ERR_UNSUPPORTED, "an fp8 KV cache needs bf16 weights");
  if (d->max_positions < 16 || d->max_positions > 65536) return laser_fail(LASER_ERR_UNSUPPORTED, "max_positions out of range");
  if (!(d->rope_theta > 1.0f) || !(d->rms_eps > 0.0f)) return laser_fail(LASER_ERR_INVALID_ARG, "bad rope_theta or rms_eps");
  return LASER_OK;
}

static laser_model* model_of(laser_model* m) { return handle_live(m) ? m : nullptr; }

// Scratch of laser_decode_step_static: a file-scope device array, one per GPU the library runs
// on, held until the process ends.  On the host its name is only a stand-in: the device
// address comes from hipGetSymbolAddress with the device current, once per device.
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
static std::mutex g_scratch_mu;
static void* g_scratch_addr[kMaxDevices];

static laser_status static_scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return laser_fail(LASER_ERR_UNSUPPORTED, "device %d (at most %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    int cur = -1;
    HIP_TRY(hipGetDevice(&cur));
    if (cur != dev) HIP_TRY(hipSetDevice(dev));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p)
      return laser_fail(LASER_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return LASER_OK;
}

}  // namespace

extern "C" laser_status laser_model_create(const laser_model_desc* desc, laser_model** out) {
  laser_status st = check_desc(desc);
  if (st != LASER_OK) return st;
  if (!out) return laser_fail(LASER_ERR_INVALID_ARG, "out is NULL");
  laser_model* m = new (std::nothrow) laser_model();
  if (!m) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  m->desc = *desc;
  m->es = desc->dtype == LASER_DTYPE_BF16 ? 2 : 4;
  m->kv_fp8 = desc->kv_dtype == LASER_DTYPE_FP8_E4M3;
  m->kv_es = m->kv_fp8 ? 1 : m->es;
  m->layers.assign(desc->n_layers, LayerW{});
  (void)hipGetDevice(&m->device);
  {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, m->device) == hipSuccess && cus > 0) m->cus = cus;
  }
  handle_add(m);
  *out = m;
  return LASER_OK;
}

extern "C" laser_status laser_model_set_tensor(laser_model* m, const char* name, const void* d_ptr, size_t bytes) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (m->finalized) return laser_fail(LASER_ERR_STATE, "model already finalized");
  if (!name || !d_ptr) return laser_fail(LASER_ERR_INVALID_ARG, "NULL name or pointer");
  const laser_model_desc& d = m->desc;
  const size_t es = m->es, D = d.d_model, hq = d.n_q_heads * (size_t)d.head_dim, hk = d.n_kv_heads * (size_t)d.head_dim;
  const void** slot = nullptr;
  size_t want = 0;
  std::string n(name);
  if (n == "embed") {
    slot = &m->embed;
    want = (size_t)d.vocab * D;
  } else if (n == "lm_head") {
    if (d.tied_embeddings) return laser_fail(LASER_ERR_INVALID_ARG, "lm_head given for a tied model");
    slot = &m->lm_head;
    want = (size_t)d.vocab * D;
  } else if (n == "final_norm") {
    slot = &m->final_norm;
    want = D;
  } else if (n.rfind("layers.", 0) == 0) {
    size_t dot = n.find('.', 7);
    if (dot == std::string::npos) return laser_fail(LASER_ERR_INVALID_ARG, "bad tensor name '%s'", name);
    int li = -1;
    try {
      li = std::stoi(n.substr(7, dot - 7));
    } catch (...) {
      li = -1;
    }
    if (li < 0 || li >= d.n_layers) return laser_fail(LASER_ERR_INVALID_ARG, "layer index out of range in '%s'", name);
    std::string f = n.substr(dot + 1);
    LayerW& L = m->layers[li];
    struct {
      const char* nm;
      const void** p;
      size_t sz;
      bool bias;
    } tab[] = {{"attn_norm", &L.attn_norm, D, false}, {"wq", &L.wq, hq * D, false}, {"wk", &L.wk, hk * D, false},
               {"wv", &L.wv, hk * D, false},         {"bq", &L.bq, hq, true},       {"bk", &L.bk, hk, true},
               {"bv", &L.bv, hk, true},              {"wo", &L.wo, D * hq, false},  {"mlp_norm", &L.mlp_norm, D, false},
               {"w_gate", &L.w_gate, (size_t)d.d_ffn * D, false}, {"w_up", &L.w_up, (size_t)d.d_ffn * D, false},
               {"w_down", &L.w_down, D * d.d_ffn, false}};
    for (auto& t : tab)
      if (f == t.nm) {
        if (t.bias && !d.qkv_bias) return laser_fail(LASER_ERR_INVALID_ARG, "bias '%s' given for a model without qkv_bias", name);
        slot = t.p;
        want = t.sz;
      }
  }
  if (!slot) return laser_fail(LASER_ERR_INVALID_ARG, "unknown tensor name '%s'", name);
  if (bytes != want * es) return laser_fail(LASER_ERR_INVALID_ARG, "'%s': %zu bytes given, %zu expected", name, bytes, want * es);
  *slot = d_ptr;
  return LASER_OK;
}

extern "C" laser_status laser_workspace_size(const laser_model* m, int max_rows, size_t* bytes) {
  if (!handle_live(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!bytes) return laser_fail(LASER_ERR_INVALID_ARG, "bytes is NULL");
  if (max_rows < 1 || max_rows > kMaxRows) return laser_fail(LASER_ERR_INVALID_ARG, "max_rows must be in [1, %d]", kMaxRows);
  *bytes = make_layout(m->desc, max_rows).total;
  return LASER_OK;
}

extern "C" laser_status laser_model_finalize(laser_model* m, int max_rows, void* d_workspace, size_t bytes, void* stream) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (m->finalized) return laser_fail(LASER_ERR_STATE, "model already finalized");
  if (max_rows < 1 || max_rows > kMaxRows) return laser_fail(LASER_ERR_INVALID_ARG, "max_rows must be in [1, %d]", kMaxRows);
  const laser_model_desc& d = m->desc;
  if (!m->embed || !m->final_norm || (!d.tied_embeddings && !m->lm_head))
    return laser_fail(LASER_ERR_STATE, "embed / final_norm / lm_head not set");
  for (int i = 0; i < d.n_layers; ++i) {
    const LayerW& L = m->layers[i];
    if (!L.attn_norm || !L.wq || !L.wk || !L.wv || !L.wo || !L.mlp_norm || !L.w_gate || !L.w_up || !L.w_down ||
        (d.qkv_bias && (!L.bq || !L.bk || !L.bv)))
      return laser_fail(LASER_ERR_STATE, "layer %d has unset tensors", i);
  }
  Layout L = make_layout(d, max_rows);
  if (!d_workspace || bytes < L.total) return laser_fail(LASER_ERR_INVALID_ARG, "workspace of %zu bytes needed", L.total);
  if (L.attn_part_bytes >= (1ull << 31))  // read by buffer instructions with 32-bit offsets
    return laser_fail(LASER_ERR_UNSUPPORTED, "attention partials of %zu bytes exceed 2 GiB", L.attn_part_bytes);
  hipStream_t s = (hipStream_t)stream;
  // RoPE table: angle pos * theta^(-2i/hd), computed in double precision
  const int half = d.head_dim / 2;
  std::vector<float2> rope((size_t)d.max_positions * half);
  for (int p = 0; p < d.max_positions; ++p)
    for (int i = 0; i < half; ++i) {
      const double ang = (double)p * std::pow((double)d.rope_theta, -2.0 * i / d.head_dim);
      rope[(size_t)p * half + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
    }
  Plan* hp = nullptr;
  // fine-grained: the forward's first kernel reads the staged plan over the bus, uncached
  HIP_TRY(hipHostMalloc((void**)&hp, sizeof(Plan) * kRing, hipHostMallocCoherent));
  for (int i = 0; i < kRing; ++i) {
    hipError_t e = hipEventCreateWithFlags(&m->ring_ev[i], hipEventDisableTiming);
    if (e != hipSuccess) {
      for (int j = 0; j < i; ++j) (void)hipEventDestroy(m->ring_ev[j]);
      (void)hipHostFree(hp);
      return laser_fail(LASER_ERR_HIP, "hipEventCreate: %s", hipGetErrorString(e));
    }
  }
  hipStream_t cs = nullptr;
  {
    hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
    if (e != hipSuccess) {
      for (int j = 0; j < kRing; ++j) (void)hipEventDestroy(m->ring_ev[j]);
      (void)hipHostFree(hp);
      return laser_fail(LASER_ERR_HIP, "hipStreamCreate: %s", hipGetErrorString(e));
    }
  }
  m->cap_stream = cs;
  char* ws = (char*)d_workspace;
  HIP_TRY(hipMemcpyAsync(ws + L.rope, rope.data(), rope.size() * sizeof(float2), hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemsetAsync(ws + L.attn_cnt, 0, L.attn_cnt_bytes, s));
  HIP_TRY(hipMemsetAsync(ws + L.kcnt, 0, L.kcnt_bytes, s));
  HIP_TRY(hipMemsetAsync(ws + L.mcnt, 0, L.mcnt_bytes, s));
  HIP_TRY(hipStreamSynchronize(s));  // the host rope table goes out of scope
  m->static_plan = new (std::nothrow) Plan;
  if (static_scratch_address(m->device, &m->static_scratch) != LASER_OK) m->static_scratch = nullptr;
  laser_clear_error();  // (the static entry point reports a missing address when called)
  m->ws = ws;
  m->lay = L;
  m->h_plans = hp;
  m->max_rows = max_rows;
  m->finalized = true;
  return LASER_OK;
}

// ----------------------------------------------------------------------------- weight tiles

namespace {
// One projection's MFMA-path geometry: 16-row groups over K columns, and its tile bytes.
struct TileProj {
  int epi, groups, K;
  size_t bytes(int es) const { return (size_t)groups * ((K + 31) / 32) * 1024 * (es / 2); }
};
TileProj tile_qkv(const laser_model_desc& d) {
  return {EPI_QKV, proj_groups(EPI_QKV, (d.n_q_heads + 2 * d.n_kv_heads) * d.head_dim, 16), d.d_model};
}
TileProj tile_o(const laser_model_desc& d) { return {EPI_RESID, proj_groups(EPI_RESID, d.d_model, 16), d.n_q_heads * d.head_dim}; }
TileProj tile_gu(const laser_model_desc& d) { return {EPI_SWIGLU, proj_groups(EPI_SWIGLU, 2 * d.d_ffn, 16), d.d_model}; }
TileProj tile_down(const laser_model_desc& d) { return {EPI_RESID, proj_groups(EPI_RESID, d.d_model, 16), d.d_ffn}; }
TileProj tile_lm(const laser_model_desc& d) { return {EPI_LMHEAD, groups_lm(d, 16), d.d_model}; }

size_t tile_total(const laser_model* m) {
  const laser_model_desc& d = m->desc;
  const size_t per_layer = tile_qkv(d).bytes(m->es) + tile_o(d).bytes(m->es) + tile_gu(d).bytes(m->es) +
                           tile_down(d).bytes(m->es);
  return per_layer * d.n_layers + tile_lm(d).bytes(m->es);
}

void drop_graphs(laser_model* m) {
  for (auto& g : m->graphs) release_graph(g);
  m->graphs.clear();
}
}  // namespace

extern "C" laser_status laser_model_tile_bytes(const laser_model* m, size_t* bytes) {
  if (!handle_live(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!bytes) return laser_fail(LASER_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = tile_total(m);
  return LASER_OK;
}

extern "C" laser_status laser_model_set_tiles(laser_model* m, void* d_buf, size_t bytes, void* stream) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!m->finalized) return laser_fail(LASER_ERR_STATE, "model not finalized");
  if (!d_buf) {  // back to the row-major tensors
    m->tiles_on = false;
    drop_graphs(m);
    return LASER_OK;
  }
  if (bytes < tile_total(m)) return laser_fail(LASER_ERR_INVALID_ARG, "tile buffer of %zu bytes needed", tile_total(m));
  const laser_model_desc& d = m->desc;
  const int dt = d.dtype == LASER_DTYPE_BF16 ? 1 : 0;
  hipStream_t s = (hipStream_t)stream;
  char* p = (char*)d_buf;
  GemmArgs base{};
  base.hq = d.n_q_heads;
  base.hkv = d.n_kv_heads;
  base.hd = d.head_dim;
  base.F = d.d_ffn;
  auto tile = [&](const TileProj& tp, GemmArgs a, int N) -> const char* {
    a.K = tp.K;
    a.N = N;
    a.n_groups = tp.groups;
    const hipError_t e = launch_tile_weights(dt, tp.epi, a, p, s);
    if (e != hipSuccess) return nullptr;
    const char* out = p;
    p += tp.bytes(m->es);
    return out;
  };
  std::vector<laser_model::Tiles> tiles(d.n_layers);
  for (int li = 0; li < d.n_layers; ++li) {
    const LayerW& W = m->layers[li];
    GemmArgs a = base;
    a.w0 = W.wq;
    a.w1 = W.wk;
    a.w2 = W.wv;
    tiles[li].qkv = tile(tile_qkv(d), a, (d.n_q_heads + 2 * d.n_kv_heads) * d.head_dim);
    a = base;
    a.w0 = W.wo;
    tiles[li].o = tile(tile_o(d), a, d.d_model);
    a = base;
    a.w0 = W.w_gate;
    a.w1 = W.w_up;
    tiles[li].gu = tile(tile_gu(d), a, 2 * d.d_ffn);
    a = base;
    a.w0 = W.w_down;
    tiles[li].down = tile(tile_down(d), a, d.d_model);
    if (!tiles[li].qkv || !tiles[li].o || !tiles[li].gu || !tiles[li].down)
      return laser_fail(LASER_ERR_HIP, "weight tiles: %s", hipGetErrorString(hipGetLastError()));
  }
  GemmArgs a = base;
  a.w0 = d.tied_embeddings ? m->embed : m->lm_head;
  const char* lm = tile(tile_lm(d), a, d.vocab);
  if (!lm) return laser_fail(LASER_ERR_HIP, "weight tiles: %s", hipGetErrorString(hipGetLastError()));
  m->tiles = std::move(tiles);
  m->lm_tile = lm;
  m->tiles_on = true;
  drop_graphs(m);
  return LASER_OK;
}

extern "C" laser_status laser_model_destroy(laser_model* m) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  handle_del(m);
  if (m->finalized) {
    (void)hipDeviceSynchronize();  // forwards still queued read the staging ring (events mark only some)
    for (int i = 0; i < kRing; ++i) (void)hipEventDestroy(m->ring_ev[i]);
    (void)hipHostFree(m->h_plans);
    for (auto& g : m->graphs) release_graph(g);
    if (m->cap_stream) (void)hipStreamDestroy(m->cap_stream);
  }
  for (auto e : m->ev_pool) (void)hipEventDestroy(e);
  delete m->static_plan;
  delete m;
  return LASER_OK;
}

// ----------------------------------------------------------------------------- KV cache

extern "C" laser_status laser_kv_pool_bytes(const laser_model* m, int num_pages, size_t* bytes_per_pool) {
  if (!handle_live(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!bytes_per_pool || num_pages < 1) return laser_fail(LASER_ERR_INVALID_ARG, "bad argument");
  const laser_model_desc& d = m->desc;
  *bytes_per_pool = (size_t)d.n_layers * num_pages * d.n_kv_heads * kPage * d.head_dim * m->kv_es;
  return LASER_OK;
}

extern "C" laser_status laser_kv_create(const laser_model* m, int num_pages, int max_seqs, int max_pages_per_seq,
                                        void* d_k_pool, void* d_v_pool, int32_t* d_block_table, laser_kv** out) {
  if (!handle_live(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!out || !d_k_pool || !d_v_pool || !d_block_table) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (num_pages < 1 || max_seqs < 1 || max_pages_per_seq < 1)
    return laser_fail(LASER_ERR_INVALID_ARG, "sizes must be positive");
  if ((long long)max_pages_per_seq * kPage > m->desc.max_positions + kPage)
    return laser_fail(LASER_ERR_INVALID_ARG, "max_pages_per_seq exceeds max_positions");
  laser_kv* kv = new (std::nothrow) laser_kv(m, num_pages, max_seqs, max_pages_per_seq, d_k_pool, d_v_pool, d_block_table);
  if (!kv) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  handle_add(kv);
  *out = kv;
  return LASER_OK;
}

static laser_kv* kv_of(const laser_kv* kv) { return handle_live(kv) ? const_cast<laser_kv*>(kv) : nullptr; }

extern "C" laser_status laser_kv_add_seq(laser_kv* kv, int seq_id, int length) {
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  if (length > kv->m->desc.max_positions) return laser_fail(LASER_ERR_INVALID_ARG, "length exceeds max_positions");
  return (laser_status)kv->pool.add_seq(seq_id, length, &kv->pending);
}

extern "C" laser_status laser_kv_free_seq(laser_kv* kv, int seq_id) {
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  return (laser_status)kv->pool.free_seq(seq_id);
}

extern "C" laser_status laser_kv_seq_len(const laser_kv* kv, int seq_id, int* len_out) {
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  if (!len_out) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (!kv->pool.live(seq_id)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq_id);
  *len_out = kv->pool.len(seq_id);
  return LASER_OK;
}

extern "C" laser_status laser_kv_page_table(const laser_kv* kv, int seq_id, int32_t* out, int cap, int* n_out) {
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  if (!out || !n_out) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (!kv->pool.live(seq_id)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq_id);
  const auto& t = kv->pool.table(seq_id);
  if ((int)t.size() > cap) return laser_fail(LASER_ERR_INVALID_ARG, "cap %d < %d pages", cap, (int)t.size());
  for (size_t i = 0; i < t.size(); ++i) out[i] = t[i];
  *n_out = (int)t.size();
  return LASER_OK;
}

extern "C" laser_status laser_kv_destroy(laser_kv* kv) {
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  handle_del(kv);
  delete kv;
  return LASER_OK;
}

// ----------------------------------------------------------------------------- launches

namespace {

struct Launch {
  laser_model* m;
  hipStream_t s;
};

// Timing session: while any class is enabled, forwards launch kernel by kernel and every
// launch records a fence-free event at its end (`next_stop`).  A class's launch then spans
// from the end of the kernel launched just before it to the end of its own last kernel;
// with kernels running back to back this equals the sum of their kernel-trace durations.
static hipEvent_t next_timing_event(void* ctx) {
  laser_model* m = (laser_model*)ctx;
  if (m->ev_used >= kMaxTimingEvents) return nullptr;
  if (m->ev_used == (int)m->ev_pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    m->ev_pool.push_back(e);
  }
  m->last_stop = m->ev_used;
  return m->ev_pool[m->ev_used++];
}

static bool timing_session(const laser_model* m) {
  for (const auto& t : m->timers)
    if (t.enabled) return true;
  return false;
}

// Arms the end-of-launch events for the current thread while a forward is being launched.
struct TimingScope {
  LaunchEvents saved;
  explicit TimingScope(laser_model* m) : saved(launch_events()) {
    if (timing_session(m)) {
      launch_events().next_stop = next_timing_event;
      launch_events().ctx = m;
    }
  }
  ~TimingScope() { launch_events() = saved; }
};

template <class F>
static hipError_t timed(laser_model* m, int cls, hipStream_t s, F&& f) {
  (void)s;
  Timer& t = m->timers[cls];
  if (!t.enabled) return f();
  const int before = m->last_stop;
  hipError_t e = f();
  if (e == hipSuccess && before >= 0 && m->last_stop != before) t.spans.emplace_back(before, m->last_stop);
  return e;
}

// Copies the used part of a plan into the next pinned staging slot, once the forward that
// last used the slot has finished (slots are taken in turn; the event recorded after the last
// slot of each block of kRingEventEvery is awaited before the block's first slot is reused).  The forward's first kernel (k_plan_fetch) copies it on to
// the device plan slot, so a replayed forward is one graph launch with no copy command before
// it (a host-to-device copy between graph launches cost about 20 us of idle time per step).
// staged_done marks the slot in use until the work now on the stream has finished.
static laser_status stage_plan(laser_model* m, const Plan& p, const Plan** hp_out, int* slot_out) {
  const int slot = m->ring_pos;
  m->ring_pos = (m->ring_pos + 1) % kRing;
  if (slot == 0) ++m->ring_turn;
  const int last = slot + kRingEventEvery - 1;  // the block's last slot
  if (slot % kRingEventEvery == 0 && m->ring_turn > 1) {
    // the block was last used in the previous turn; its last forward's event covers it (one
    // stream per model), unless that forward failed before its event was recorded
    if (m->ring_used[last] && m->ring_rec_turn[last] == m->ring_turn - 1)
      HIP_TRY(hipEventSynchronize(m->ring_ev[last]));
    else
      HIP_TRY(hipDeviceSynchronize());
  }
  Plan* hp = m->h_plans + slot;
  std::memcpy(hp, &p, offsetof(Plan, items) + sizeof(AttnItem) * (size_t)p.n_items);
  std::memcpy(hp->bt, p.bt, sizeof(BtUpdate) * (size_t)p.n_bt);
  *hp_out = hp;
  *slot_out = slot;
  return LASER_OK;
}

static laser_status staged_done(laser_model* m, int slot, hipStream_t s) {
  if (slot % kRingEventEvery != kRingEventEvery - 1) return LASER_OK;
  HIP_TRY(hipEventRecord(m->ring_ev[slot], s));
  m->ring_used[slot] = true;
  m->ring_rec_turn[slot] = m->ring_turn;
  return LASER_OK;
}

// Sends block-table writes that are not part of a forward plan (after add_seq).
// (buf: a host plan buffer to build in; NULL: one is allocated per upload)
static laser_status flush_pending(laser_kv* kv, laser_model* m, hipStream_t s, Plan* buf = nullptr) {
  size_t i = 0;
  while (i < kv->pending.size()) {
    Plan* p = buf ? buf : new (std::nothrow) Plan;
    if (!p) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
    p->M = p->n_groups = p->n_out = p->n_items = 0;
    p->n_bt = 0;
    while (i < kv->pending.size() && p->n_bt < kMaxBt) {
      const PageUpdate& u = kv->pending[i++];
      p->bt[p->n_bt++] = BtUpdate{u.seq, u.idx, u.page};
    }
    const Plan* hp = nullptr;
    int slot = 0;
    laser_status st = stage_plan(m, *p, &hp, &slot);
    if (!buf) delete p;
    if (st != LASER_OK) return st;
    Plan* dp = m->wsp<Plan>(m->lay.plans);  // stream order keeps forwards off each other's plan
    TimingScope scope(m);
    HIP_TRY(launch_plan_fetch(hp, dp, s));
    HIP_TRY(launch_apply_bt(dp, kv->bt, kv->pool.max_pages_per_seq(), s));
    st = staged_done(m, slot, s);
    if (st != LASER_OK) return st;
  }
  kv->pending.clear();
  return LASER_OK;
}

// Row groups, their attention splits and the attention work items.  Rows come in runs of one
// sequence (spans).  Runs whose sequences start with the same page are a request and its
// forks: they share their leading full pages, so one group over those pages holds the rows
// of all of them (each shared page is read once for every row), and each run keeps a group
// of its own for its later pages.  A row's partials from the two are merged like any split.
// The rows are reordered so that a family's runs are contiguous (outputs follow their rows).
static void plan_groups(const laser_model* m, const laser_kv* kv, Plan& p) {
  const laser_model_desc& d = m->desc;
  const int G = d.n_q_heads / d.n_kv_heads;
  struct Run {
    int seq, r0, r1, family;
  };
  std::vector<Run> runs;
  for (int r = 0; r < p.M;) {
    int e = r + 1;
    while (e < p.M && p.rows[e].seq == p.rows[r].seq) ++e;
    runs.push_back({p.rows[r].seq, r, e, -1});
    r = e;
  }
  struct Family {
    std::vector<int> members;  // runs
    int shared;                // leading full pages shared by every member (0: none)
  };
  std::vector<Family> fams;
  for (size_t i = 0; i < runs.size(); ++i) {
    if (runs[i].family >= 0) continue;
    const std::vector<int>& ti = kv->pool.table(runs[i].seq);
    runs[i].family = (int)fams.size();
    Family f{{(int)i}, 0};
    for (size_t j = i + 1; j < runs.size() && !ti.empty(); ++j) {
      const std::vector<int>& tj = kv->pool.table(runs[j].seq);
      if (runs[j].family < 0 && !tj.empty() && tj[0] == ti[0]) {
        runs[j].family = (int)fams.size();
        f.members.push_back((int)j);
      }
    }
    if (f.members.size() > 1) {
      int sh = (int)ti.size();
      for (int k : f.members) {
        const std::vector<int>& t = kv->pool.table(runs[k].seq);
        int n = 0, minpos = p.rows[runs[k].r0].pos;
        while (n < (int)t.size() && n < (int)ti.size() && t[n] == ti[n]) ++n;
        for (int r = runs[k].r0; r < runs[k].r1; ++r) minpos = std::min(minpos, p.rows[r].pos);
        // only pages wholly below the run's first position (every row sees all of them)
        sh = std::min(sh, std::min(n, minpos / kPage));
      }
      f.shared = sh;
    }
    fams.push_back(f);
  }
  // family by family, runs in their order
  std::vector<int> order, newrow(p.M);
  for (const Family& f : fams)
    for (int k : f.members)
      for (int r = runs[k].r0; r < runs[k].r1; ++r) {
        newrow[r] = (int)order.size();
        order.push_back(r);
      }
  bool moved = false;
  for (int i = 0; i < p.M; ++i) moved |= order[i] != i;
  if (moved) {
    std::vector<RowDesc> old(p.rows, p.rows + p.M);
    for (int i = 0; i < p.M; ++i) p.rows[i] = old[order[i]];
    for (int o = 0; o < p.n_out; ++o) p.outs[o].row = newrow[p.outs[o].row];
    for (Run& rn : runs) {
      const int n = rn.r1 - rn.r0;
      rn.r0 = newrow[rn.r0];
      rn.r1 = rn.r0 + n;
    }
  }

  p.n_groups = 0;
  std::vector<int> row_prefix(p.M, -1), row_own(p.M, -1);
  auto add_group = [&](int seq, int r0, int r1, int pbeg, bool prefix) {
    int maxpos = 0;
    for (int q = r0; q < r1; ++q) maxpos = std::max(maxpos, p.rows[q].pos);
    const int gi = p.n_groups++;
    GroupDesc& g = p.groups[gi];
    g.seq = seq;
    g.row0 = r0;
    g.nrows = r1 - r0;
    g.pbeg = pbeg;
    g.npages = prefix ? pbeg : maxpos / kPage + 1;  // (a prefix group's end is set by its caller)
    g.maxpos = maxpos;
    g.slot0 = 0;
    g.direct = 0;
    g.fused = 0;
    for (int q = r0; q < r1; ++q) (prefix ? row_prefix : row_own)[q] = gi;
    return gi;
  };
  for (const Family& f : fams) {
    if (f.shared > 0) {  // the rows of all members over the shared pages
      const int gi = add_group(runs[f.members[0]].seq, runs[f.members[0]].r0, runs[f.members.back()].r1, 0, true);
      p.groups[gi].npages = f.shared;
    }
    for (int k : f.members) add_group(runs[k].seq, runs[k].r0, runs[k].r1, f.shared, false);  // own pages
  }
  // A work item (workgroup) takes one 16-column query tile of a group and spreads a split of
  // its pages over its 4 waves.  Splits of at most kMaxPagesPerWave pages per wave, enough
  // of them to give about kTargetAttnWaves waves; a group of several tiles lists its splits
  // in chunks of 8, tile by tile, so that the tiles of one split are 8 items apart (workgroups
  // go to the 8 XCDs in turn: they share one XCD's L2).  Partial slots of a row: its
  // shared-pages group's splits, then its own group's; own groups next to a shared one get at
  // most kOwnSlots splits.
  auto ntiles = [&](const GroupDesc& g) { return ceil_div(g.nrows * G, 16); };
  long long units = 0;
  for (int i = 0; i < p.n_groups; ++i)
    units += (long long)(p.groups[i].npages - p.groups[i].pbeg) * d.n_kv_heads * ntiles(p.groups[i]);
  constexpr int kOwnSlots = 8;
  int base = std::min(kMaxPagesPerWave, std::max(1, (int)((units + kTargetAttnWaves - 1) / kTargetAttnWaves)));
  auto item_count = [&]() {
    int n = 0;
    for (int i = 0; i < p.n_groups; ++i) {
      const GroupDesc& g = p.groups[i];
      const int T = ntiles(g);
      n = (T == 1 || g.nwg < 8) ? n + g.nwg * T : ceil_div(n, 8) * 8 + ceil_div(g.nwg, 8) * 8 * T;
    }
    return n;
  };
  // one-row groups with no shared-prefix group can merge their own splits (fewer, longer ones)
  auto fusable = [&](const GroupDesc& g) { return m->attn_fuse && g.nrows == 1 && row_prefix[g.row0] < 0; };
  for (;; base *= 2) {  // (more pages per wave only if the items would not fit)
    for (int i = 0; i < p.n_groups; ++i) {
      GroupDesc& g = p.groups[i];
      const bool shares = row_prefix[g.row0] >= 0;
      const bool is_prefix = row_prefix[g.row0] == i;
      const int max_wg = fusable(g) ? m->attn_fuse_max
                                    : is_prefix ? kAttnMaxWG - kOwnSlots : (shares ? kOwnSlots : kAttnMaxWG);
      const int npg = g.npages - g.pbeg;
      g.pps = std::max(base, ceil_div(npg, max_wg * kAttnWaves));
      g.nwg = ceil_div(npg, kAttnWaves * g.pps);
    }
    if (item_count() <= kMaxAttnItems) break;
  }
  for (int i = 0; i < p.n_groups; ++i) {
    GroupDesc& g = p.groups[i];
    const int pre = row_prefix[g.row0];
    if (pre >= 0 && pre != i) g.slot0 = p.groups[pre].nwg;
    g.direct = pre < 0 && g.nwg == 1;
    g.fused = !g.direct && fusable(g);
  }
  // (a fused row counts as written directly: the merge kernel skips it)
  for (int q = 0; q < p.M; ++q)
    p.row_nslots[q] = p.groups[row_own[q]].fused
                          ? 1
                          : p.groups[row_own[q]].nwg + (row_prefix[q] >= 0 ? p.groups[row_prefix[q]].nwg : 0);

  p.n_items = 0;
  auto push = [&](const GroupDesc* g, int wg, int tile) {
    AttnItem& it = p.items[p.n_items++];
    if (!g) {
      it = AttnItem{0, 0, 0, 0, 0, 0, 0, 0};
      return;
    }
    it.seq = g->seq;
    it.row0 = g->row0;
    it.nrows = g->nrows | (g->fused ? g->nwg << 8 | (int)(g - p.groups) << 16 : 0);
    it.p0 = g->pbeg + wg * kAttnWaves * g->pps;
    it.pend = g->npages;
    it.pps = g->pps;
    it.maxpos = g->maxpos;
    it.info = tile | (g->slot0 + wg) << 8 | (g->direct ? 1 << 24 : 0);
  };
  for (int i = 0; i < p.n_groups; ++i) {
    const GroupDesc& g = p.groups[i];
    const int T = ntiles(g);
    if (T == 1 || g.nwg < 8) {
      for (int t = 0; t < T; ++t)
        for (int wg = 0; wg < g.nwg; ++wg) push(&g, wg, t);
      continue;
    }
    while (p.n_items % 8) push(nullptr, 0, 0);
    for (int c = 0; c < g.nwg; c += 8)
      for (int t = 0; t < T; ++t)
        for (int j = 0; j < 8; ++j) push(c + j < g.nwg ? &g : nullptr, c + j, t);
  }
}

// Pads the work items with empty ones up to n (the grid width of the launch).
static void pad_items(Plan& p, int n) {
  while (p.n_items < n) p.items[p.n_items++] = AttnItem{0, 0, 0, 0, 0, 0, 0, 0};
}

// Where a forward's scratch lives: attention partials (rows laid out for `rows` rows),
// split statistics, fused-merge arrival counters, LM-head statistics, K-share partials.
struct Scratch {
  float *attn_part, *attn_ml, *kpart;
  unsigned* kcnt;  // K-share arrival counters
  unsigned* mcnt;  // merge counters of the O-projection's launch (null: the merge kernel is used)
  float *qpart, *sqpart;  // QKV K-slice partials (null: that kernel is not used)
  unsigned* attn_cnt;
  LmPart* lm_part;
  size_t part_bytes, ml_bytes;
  int rows;
};

// The model workspace's scratch (every entry point but laser_decode_step_static).
static Scratch workspace_scratch(const laser_model* m) {
  const Layout& L = m->lay;
  return Scratch{m->wsp<float>(L.attn_part),
                 m->wsp<float>(L.attn_ml),
                 m->wsp<float>(L.kpart),
                 m->wsp<unsigned>(L.kcnt),
                 m->wsp<unsigned>(L.mcnt),
                 L.qpart ? m->wsp<float>(L.qpart) : nullptr,
                 L.sqpart ? m->wsp<float>(L.sqpart) : nullptr,
                 m->wsp<unsigned>(L.attn_cnt), m->wsp<LmPart>(L.lm_part), L.attn_part_bytes, L.attn_ml_bytes,
                 m->max_rows};
}

static laser_status launch_forward(laser_model* m, laser_kv* kv, const FwdKey& key, hipStream_t s, const Scratch& sc,
                                   const Plan* hp);

// Runs one forward: plans the attention splits, stages the plan, then launches the
// forward's kernels (replaying a captured graph of them when graphs are on and no kernel
// class is being timed).
static laser_status run_forward(laser_model* m, laser_kv* kv, Plan& p, const PlanIO& io, hipStream_t s,
                                bool allow_graph = true, const Scratch* sc_in = nullptr) {
  const Scratch sc = sc_in ? *sc_in : workspace_scratch(m);
  plan_groups(m, kv, p);
  p.io = io;
  FwdKey key{};
  key.M = p.M;
  key.n_out = p.n_out;
  int max_slots = 1;
  bool merge = false;
  for (int i = 0; i < p.n_groups; ++i) merge |= !p.groups[i].direct && !p.groups[i].fused;
  for (int q = 0; q < p.M; ++q) max_slots = std::max(max_slots, p.row_nslots[q]);
  // the merge's slot bound is rounded up so that a growing context keeps the same key for a
  // while (the merge reads the row's own count)
  key.mslots = std::min(kAttnMaxWG, ceil_div(max_slots, 8) * 8);
  key.merge = merge;
  const laser_model_desc& d = m->desc;
  key.mo = merge && sc.mcnt != nullptr && p.M <= kValuMaxRows && (d.head_dim == 64 || d.head_dim == 128) &&
           (m->oproj_merge == 2 ||
            (m->oproj_merge == 1 && (size_t)d.d_model * d.n_q_heads * d.head_dim * m->es >= kMergeMinOBytes));
  key.kv_id = kv->id;
  // The merge in the O-projection's launch: every layer's counter grows by the forward's
  // merge workgroups, and the O-projection waits for the running total.  After a forward that
  // failed part way the counters no longer match it, so they are cleared first.
  struct Resync {
    laser_model* m;
    bool armed;
    ~Resync() {
      if (armed) m->merge_resync = true;
    }
  } resync{m, false};
  if (key.mo) {
    if (m->merge_resync) {
      HIP_TRY(launch_fill_u32(sc.mcnt, (int)(m->lay.mcnt_bytes / 4), 0u, s));
      m->merge_cum = 0;
      m->merge_resync = false;
    }
    m->merge_cum += (unsigned)(p.M * d.n_q_heads);
    resync.armed = true;
  }
  p.merge_target = m->merge_cum;
  // The attention grid is at least the item count, a multiple of 8 (so that item i runs on
  // XCD i mod 8), padded with empty items.  A captured forward of the same shape whose grid
  // is at most 1/4 (+8) wider is reused; a new one is captured 1/8 wider, so a growing
  // context or a changing mix of probes does not recapture at every step.
  const int need = std::max(8, ceil_div(p.n_items, 8) * 8);
  const bool timing = timing_session(m);
  const bool graphs = allow_graph && m->use_graphs && !timing;
  GraphEntry* ge = nullptr;
  if (graphs)
    for (auto& g : m->graphs)
      if (g.key.same_shape(key) && g.key.agx >= need && g.key.agx <= need + need / 4 + 8 &&
          (!ge || g.key.agx < ge->key.agx))
        ge = &g;
  key.agx = ge ? ge->key.agx : graphs ? std::min(kMaxAttnItems, ceil_div(need + need / 8, 8) * 8) : need;
  pad_items(p, key.agx);
  const Plan* hp = nullptr;
  int slot = 0;
  laser_status st = stage_plan(m, p, &hp, &slot);
  if (st != LASER_OK) return st;
  if (!graphs) {
    {
      TimingScope scope(m);
      st = launch_forward(m, kv, key, s, sc, hp);
    }
    resync.armed = resync.armed && st != LASER_OK;
    const laser_status sd = staged_done(m, slot, s);
    return st != LASER_OK ? st : sd;
  }

  if (!ge) {
    hipGraph_t graph = nullptr;
    HIP_TRY(hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeThreadLocal));
    st = launch_forward(m, kv, key, m->cap_stream, sc, hp);
    const hipError_t ec = hipStreamEndCapture(m->cap_stream, &graph);
    if (st != LASER_OK) {
      if (graph) (void)hipGraphDestroy(graph);
      return st;
    }
    if (ec != hipSuccess) return laser_fail(LASER_ERR_HIP, "graph capture: %s", hipGetErrorString(ec));
    // the plan copy is the one root: every other kernel follows it in stream order
    hipGraphNode_t fetch = nullptr;
    size_t n_roots = 1;
    hipKernelNodeParams fp{};
    hipGraphNodeType ty{};
    if (hipGraphGetRootNodes(graph, &fetch, &n_roots) != hipSuccess || n_roots != 1 ||
        hipGraphNodeGetType(fetch, &ty) != hipSuccess || ty != hipGraphNodeTypeKernel ||
        hipGraphKernelNodeGetParams(fetch, &fp) != hipSuccess || fp.func != plan_fetch_kernel()) {
      (void)hipGraphDestroy(graph);
      return laser_fail(LASER_ERR_HIP, "graph capture: the plan copy is not the forward's only root");
    }
    hipGraphExec_t exec = nullptr;
    const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    if (ei != hipSuccess) {
      (void)hipGraphDestroy(graph);
      return laser_fail(LASER_ERR_HIP, "graph instantiate: %s", hipGetErrorString(ei));
    }
    hipEvent_t done = nullptr;
    const hipError_t ee = hipEventCreateWithFlags(&done, hipEventDisableTiming);
    if (ee != hipSuccess) {
      (void)hipGraphExecDestroy(exec);
      (void)hipGraphDestroy(graph);
      return laser_fail(LASER_ERR_HIP, "hipEventCreate: %s", hipGetErrorString(ee));
    }
    if ((int)m->graphs.size() >= kMaxGraphs) {  // the least recently used, once its last launch is done
      auto lru = std::min_element(m->graphs.begin(), m->graphs.end(),
                                  [](const GraphEntry& x, const GraphEntry& y) { return x.last_use < y.last_use; });
      release_graph(*lru);
      m->graphs.erase(lru);
    }
    m->graphs.push_back(GraphEntry{key, exec, 0, done, 0, graph, fetch, fp});
    ++m->graph_captures;
    ge = &m->graphs.back();
  }
  ge->last_use = ++m->graph_clock;
  {  // the replay's plan copy reads this call's staging slot
    Plan* dp = m->wsp<Plan>(m->lay.plans);
    void* args[2] = {(void*)&hp, (void*)&dp};
    hipKernelNodeParams kp = ge->fetch_params;
    kp.kernelParams = args;
    kp.extra = nullptr;
    HIP_TRY(hipGraphExecKernelNodeSetParams(ge->exec, ge->fetch, &kp));
  }
  HIP_TRY(hipGraphLaunch(ge->exec, s));
  if (++ge->unrecorded >= kGraphEventEvery) {
    HIP_TRY(hipEventRecord(ge->done, s));
    ge->unrecorded = 0;
  }
  resync.armed = false;
  return staged_done(m, slot, s);
}

// Launches the kernels of one forward: the copy of its staged plan (hp) to the device plan
// slot, then the forward's kernels, which read that slot.
static laser_status launch_forward(laser_model* m, laser_kv* kv, const FwdKey& key, hipStream_t s, const Scratch& sc,
                                   const Plan* hp) {
  const laser_model_desc& d = m->desc;
  const Layout& L = m->lay;
  const int hd = d.head_dim, G = d.n_q_heads / d.n_kv_heads;
  const int dt = d.dtype == LASER_DTYPE_BF16 ? 1 : 0;
  const int max_pps = kv->pool.max_pages_per_seq();
  const Plan* dp = m->wsp<Plan>(L.plans);
  laser_status st = LASER_OK;
  float* h = m->wsp<float>(L.h);
  HIP_TRY(timed(m, LASER_K_EMBED, s, [&] {  // the plan copy (from the staging slot hp), then the embedding gather
    const hipError_t e = launch_plan_fetch(hp, m->wsp<Plan>(L.plans), s);
    return e == hipSuccess ? launch_embed(dt, dp, key.M, m->embed, d.d_model, d.vocab, h, kv->bt, max_pps, s) : e;
  }));

  GemmArgs base{};
  base.plan = dp;
  base.eps = d.rms_eps;
  base.hq = d.n_q_heads;
  base.hkv = d.n_kv_heads;
  base.hd = hd;
  base.rope = m->wsp<float2>(L.rope);
  base.q_out = m->wsp<float>(L.q);
  base.kpool = kv->kpool;
  base.vpool = kv->vpool;
  base.bt = kv->bt;
  base.max_pps = max_pps;
  base.num_pages = kv->pool.num_pages();
  base.kv_fp8 = m->kv_fp8;
  base.h = h;
  base.act = m->wsp<float>(L.act);
  base.F = d.d_ffn;

  // rows: output rows of the projection (SwiGLU: gate and up rows together)
  // tile: the projection's tile-order weights (used on the MFMA path when tiles are on)
  // mg: the split merge that produces the activation rows runs in this launch (residual
  // projection, VALU path)
  auto gemm = [&](int cls, int epi, GemmArgs a, int K, int N, int rows, int M, const char* tile,
                  const MergeArgs* mg = nullptr) -> laser_status {
    int rw = proj_rw(epi, rows, M, m->cus);
    if (epi == EPI_QKV && gemv_short_rows(K, (int)m->es, M)) rw = qkv_short_rw(rows, m->cus, rw);
    a.K = K;
    a.N = N;
    a.n_groups = proj_groups(epi, rows, rw);
    const MfmaShape ms = mfma_shape(epi, a.n_groups, M, K, (int)m->es, m->cus, m->gemm_kernel);
    a.nr = ms.nr;
    a.ksplit = ms.ks;
    a.nrw = ms.nrw;
    a.kpart = sc.kpart;
    // two K shares: the later workgroup of each block adds them (measured: the 8B batch-8
    // down projection 26.8 -> 24.6 us); four (the row-wave kernel at 49-64 rows): a reduce
    // kernel, whose last arrivers' reads of 4 shares made the riding forward slower
    a.kcnt = ms.ks == 2 ? sc.kcnt : nullptr;
    a.M = M;
    if (M <= kValuMaxRows) gemv_shape(epi, K, (int)m->es, M, a.n_groups, m->cus, a);
    if (M > kValuMaxRows && m->tiles_on) {
      a.wtile = tile;
      a.tsteps = (K + 31) / 32;
    }
    if (epi == EPI_QKV && M >= kQSliceMinRows && M <= 64 && dt == 1 && sc.qpart != nullptr && m->gemm_kernel == 0 &&
        a.n_groups * 16 == N) {
      a.tsteps = (K + 31) / 32;
      HIP_TRY(timed(m, cls, s, [&] { return launch_qkv_slices(a, sc.qpart, sc.sqpart, s); }));
      return LASER_OK;
    }
    const int mode = gemm_mode(M);
    if (mg != nullptr) {
      if (epi != EPI_RESID || mode > kValuMaxRows) return laser_fail(LASER_ERR_STATE, "merged projection off the VALU path");
      HIP_TRY(timed(m, cls, s, [&] { return launch_gemv_merged(dt, rw, a, *mg, s); }));
      return LASER_OK;
    }
    HIP_TRY(timed(m, cls, s, [&] {
      hipError_t e = launch_gemm(dt, mode, epi, rw, a, s);
      if (e == hipSuccess && a.ksplit > 1 && a.kcnt == nullptr) e = launch_ksplit_reduce(a, s);
      return e;
    }));
    return LASER_OK;
  };

  AttnArgs aa{};
  aa.plan = dp;
  aa.q = m->wsp<float>(L.q);
  aa.o = m->wsp<float>(L.o);
  aa.kpool = kv->kpool;
  aa.vpool = kv->vpool;
  aa.bt = kv->bt;
  aa.max_pps = max_pps;
  aa.num_pages = kv->pool.num_pages();
  aa.hq = d.n_q_heads;
  aa.hkv = d.n_kv_heads;
  aa.G = G;
  aa.max_rows = sc.rows;
  aa.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));
  aa.part = sc.attn_part;
  aa.ml = sc.attn_ml;
  aa.part_bytes = (uint32_t)sc.part_bytes;
  aa.ml_bytes = (uint32_t)sc.ml_bytes;
  aa.cnt = sc.attn_cnt;
  const dim3 agrid(key.agx, d.n_kv_heads);

  for (int li = 0; li < d.n_layers; ++li) {
    const LayerW& W = m->layers[li];
    GemmArgs a = base;
    a.w0 = W.wq;
    a.w1 = W.wk;
    a.w2 = W.wv;
    a.b0 = W.bq;
    a.b1 = W.bk;
    a.b2 = W.bv;
    a.x = h;
    a.ldx = d.d_model;
    a.gain = W.attn_norm;
    a.layer = li;
    const laser_model::Tiles* T = m->tiles_on ? &m->tiles[li] : nullptr;
    st = gemm(LASER_K_QKV, EPI_QKV, a, d.d_model, (d.n_q_heads + 2 * d.n_kv_heads) * hd,
              (d.n_q_heads + 2 * d.n_kv_heads) * hd, key.M, T ? T->qkv : nullptr);
    if (st != LASER_OK) return st;

    aa.layer = li;
    HIP_TRY(timed(m, LASER_K_ATTN, s, [&] {
      hipError_t e = launch_attn(m->kv_fp8 ? 2 : dt, hd, aa, agrid, s);
      if (e == hipSuccess && key.merge && !key.mo) e = launch_attn_merge(aa, key.M, hd, key.mslots, s);
      return e;
    }));

    a = base;
    a.w0 = W.wo;
    a.x = m->wsp<float>(L.o);
    a.ldx = d.n_q_heads * hd;
    a.gain = nullptr;
    MergeArgs mg{};
    if (key.mo) {
      mg.part = aa.part;
      mg.ml = aa.ml;
      mg.cnt = sc.mcnt + (size_t)li * kMgReplicas * kKsCntStride;
      mg.o_bytes = (uint32_t)((size_t)key.M * d.n_q_heads * hd * 4);
      mg.hq = d.n_q_heads;
      mg.G = G;
      mg.hd = hd;
      mg.max_rows = sc.rows;
      mg.nslots = key.mslots;
      mg.nwg = key.M * d.n_q_heads;
    }
    st = gemm(LASER_K_OPROJ, EPI_RESID, a, d.n_q_heads * hd, d.d_model, d.d_model, key.M, T ? T->o : nullptr,
              key.mo ? &mg : nullptr);
    if (st != LASER_OK) return st;

    a = base;
    a.w0 = W.w_gate;
    a.w1 = W.w_up;
    a.x = h;
    a.ldx = d.d_model;
    a.gain = W.mlp_norm;
    st = gemm(LASER_K_GATEUP, EPI_SWIGLU, a, d.d_model, 2 * d.d_ffn, 2 * d.d_ffn, key.M, T ? T->gu : nullptr);
    if (st != LASER_OK) return st;

    a = base;
    a.w0 = W.w_down;
    a.x = m->wsp<float>(L.act);
    a.ldx = d.d_ffn;
    a.gain = nullptr;
    st = gemm(LASER_K_DOWN, EPI_RESID, a, d.d_ffn, d.d_model, d.d_model, key.M, T ? T->down : nullptr);
    if (st != LASER_OK) return st;
  }
  if (key.n_out > 0) {
    GemmArgs a = base;
    a.w0 = d.tied_embeddings ? m->embed : m->lm_head;
    a.x = h;
    a.ldx = d.d_model;
    a.gain = m->final_norm;
    a.row_map = 1;
    a.lm_part = sc.lm_part;
    a.K = d.d_model;
    a.N = d.vocab;
    a.n_groups = groups_lm(d, key.n_out);
    const MfmaShape ms = mfma_shape(EPI_LMHEAD, a.n_groups, key.n_out, d.d_model, (int)m->es, m->cus, m->gemm_kernel);
    a.nr = ms.nr;
    a.nrw = ms.nrw;
    a.ksplit = 1;
    a.M = key.n_out;
    if (key.n_out <= kValuMaxRows) gemv_shape(EPI_LMHEAD, d.d_model, (int)m->es, key.n_out, a.n_groups, m->cus, a);
    if (key.n_out > kValuMaxRows && m->tiles_on) {
      a.wtile = m->lm_tile;
      a.tsteps = (d.d_model + 31) / 32;
    }
    HIP_TRY(timed(m, LASER_K_LMHEAD, s, [&] {
      hipError_t e = launch_gemm(dt, gemm_mode(key.n_out), EPI_LMHEAD, key.n_out > kValuMaxRows ? 16 : 8, a, s);
      if (e == hipSuccess) e = launch_lm_reduce(dp, a.lm_part, a.n_groups, key.n_out, s);
      return e;
    }));
  }
  return LASER_OK;
}

static laser_status check_ready(laser_model* m, laser_kv* kv) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!m->finalized) return laser_fail(LASER_ERR_STATE, "model not finalized");
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  if (kv->m != m) return laser_fail(LASER_ERR_INVALID_ARG, "kv cache belongs to another model");
  return LASER_OK;
}

// Validates that every (seq, growth) can be satisfied at once: distinct live sequences,
// positions below max_positions, pages per sequence and free pages in total.
static laser_status check_growth(laser_model* m, laser_kv* kv, const std::vector<int>& seqs, const std::vector<int>& grow) {
  std::unordered_set<int> seen;
  long long need = 0;
  for (size_t i = 0; i < seqs.size(); ++i) {
    const int sq = seqs[i];
    if (!kv->pool.live(sq)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", sq);
    if (!seen.insert(sq).second) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d repeated", sq);
    const int nl = kv->pool.len(sq) + grow[i];
    if (nl > m->desc.max_positions) return laser_fail(LASER_ERR_INVALID_ARG, "seq %d would exceed max_positions", sq);
    if (kv->pool.pages_for(nl) > kv->pool.max_pages_per_seq())
      return laser_fail(LASER_ERR_INVALID_ARG, "seq %d would exceed max_pages_per_seq", sq);
    need += kv->pool.pages_needed(sq, grow[i]);
  }
  if (need > kv->pool.num_free()) return laser_fail(LASER_ERR_OUT_OF_PAGES, "need %lld pages, %d free", need, kv->pool.num_free());
  return LASER_OK;
}

static void push_updates(Plan& p, const std::vector<PageUpdate>& u) {
  for (const auto& x : u) p.bt[p.n_bt++] = BtUpdate{x.seq, x.idx, x.page};
}

}  // namespace

extern "C" laser_status laser_kv_import(laser_kv* kv, int seq_id, const void* d_k, const void* d_v, int length, void* stream) {
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  laser_model* m = const_cast<laser_model*>(kv->m);
  if (!model_of(m) || !m->finalized) return laser_fail(LASER_ERR_STATE, "model not finalized");
  if (!d_k || !d_v) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (!kv->pool.live(seq_id)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq_id);
  if (length != kv->pool.len(seq_id)) return laser_fail(LASER_ERR_INVALID_ARG, "length %d != sequence length %d", length, kv->pool.len(seq_id));
  hipStream_t s = (hipStream_t)stream;
  laser_status st = flush_pending(kv, m, s);
  if (st != LASER_OK) return st;
  const laser_model_desc& d = m->desc;
  HIP_TRY(launch_kv_copy(m->kv_es, 1, kv->kpool, kv->vpool, kv->bt, kv->pool.max_pages_per_seq(),
                         kv->pool.num_pages(), d.n_layers, d.n_kv_heads, d.head_dim, seq_id, length,
                         const_cast<void*>(d_k), const_cast<void*>(d_v), s));
  return LASER_OK;
}

extern "C" laser_status laser_kv_export(const laser_kv* kvc, int seq_id, void* d_k, void* d_v, void* stream) {
  laser_kv* kv = kv_of(kvc);
  if (!kv) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  laser_model* m = const_cast<laser_model*>(kv->m);
  if (!model_of(m) || !m->finalized) return laser_fail(LASER_ERR_STATE, "model not finalized");
  if (!d_k || !d_v) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (!kv->pool.live(seq_id)) return laser_fail(LASER_ERR_INVALID_ARG, "seq_id %d not present", seq_id);
  hipStream_t s = (hipStream_t)stream;
  laser_status st = flush_pending(kv, m, s);
  if (st != LASER_OK) return st;
  const laser_model_desc& d = m->desc;
  HIP_TRY(launch_kv_copy(m->kv_es, 0, kv->kpool, kv->vpool, kv->bt, kv->pool.max_pages_per_seq(),
                         kv->pool.num_pages(), d.n_layers, d.n_kv_heads, d.head_dim, seq_id, kv->pool.len(seq_id), d_k, d_v, s));
  return LASER_OK;
}

extern "C" laser_status laser_decode_step(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                                          const int32_t* d_tokens, int32_t* d_next, float* d_max_prob, float* d_logits,
                                          void* stream) {
  laser_status st = check_ready(m, kv);
  if (st != LASER_OK) return st;
  if (batch < 1 || batch > m->max_rows) return laser_fail(LASER_ERR_INVALID_ARG, "batch must be in [1, %d]", m->max_rows);
  if (!seq_ids || !d_tokens || !d_next || !d_max_prob) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  std::vector<int> seqs(seq_ids, seq_ids + batch), grow(batch, 1);
  st = check_growth(m, kv, seqs, grow);
  if (st != LASER_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  st = flush_pending(kv, m, s);
  if (st != LASER_OK) return st;
  Plan* p = new (std::nothrow) Plan;
  if (!p) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  p->M = batch;
  p->n_out = batch;
  p->n_bt = 0;
  std::vector<PageUpdate> upd;
  for (int b = 0; b < batch; ++b) {
    const int pos = kv->pool.len(seqs[b]);
    kv->pool.append(seqs[b], 1, &upd);
    p->rows[b] = RowDesc{seqs[b], pos, 0, b};
    p->outs[b] = OutDesc{b, 0, b, 0};
  }
  push_updates(*p, upd);
  PlanIO io{};
  io.tok_src[0] = io.tok_src[1] = d_tokens;
  io.tok_dst[0] = d_next;
  io.p_dst[0] = d_max_prob;
  io.logits[0] = d_logits;
  st = run_forward(m, kv, *p, io, s);
  delete p;
  return st;
}

// laser_decode_step with its scratch in the static array: the same plan and kernels, launched
// one by one (no graph is captured or instantiated), the host plan built in the model's
// buffer, the arrival counters cleared by a kernel.  Allocates nothing.
extern "C" laser_status laser_decode_step_static(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                                                 const int32_t* d_tokens, int32_t* d_next, float* d_max_prob,
                                                 float* d_logits, void* stream) {
  laser_status st = check_ready(m, kv);
  if (st != LASER_OK) return st;
  if (batch < 1 || batch > m->max_rows) return laser_fail(LASER_ERR_INVALID_ARG, "batch must be in [1, %d]", m->max_rows);
  if (!seq_ids || !d_tokens || !d_next || !d_max_prob) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (!m->static_scratch || !m->static_plan)
    return laser_fail(LASER_ERR_STATE, "the static scratch array's address is unavailable on device %d", m->device);
  // scratch layout for `batch` rows
  const laser_model_desc& d = m->desc;
  const int G = d.n_q_heads / d.n_kv_heads;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t part_bytes = (size_t)d.n_kv_heads * kAttnMaxWG * batch * G * d.head_dim * 4;
  const size_t ml_bytes = (size_t)d.n_kv_heads * kAttnMaxWG * batch * G * 2 * 4;
  const size_t cnt_n = (size_t)d.n_kv_heads * kMaxGroups * kAttnCntStride;
  const size_t o_part = take(part_bytes), o_ml = take(ml_bytes), o_cnt = take(cnt_n * 4);
  const size_t o_lm = take((size_t)groups_lm(d, batch) * batch * sizeof(LmPart));
  const size_t o_kpart = take((size_t)kMaxKsplit * batch * d.d_model * 4);
  const size_t kcnt_bytes = ks_cnt_bytes(d), o_kcnt = take(kcnt_bytes);
  if (off > kStaticScratchBytes)
    return laser_fail(LASER_ERR_UNSUPPORTED, "batch %d needs %zu bytes of scratch; the static array holds %zu", batch,
                      off, kStaticScratchBytes);
  char* base = (char*)m->static_scratch;
  const Scratch sc{(float*)(base + o_part), (float*)(base + o_ml), (float*)(base + o_kpart), (unsigned*)(base + o_kcnt),
                   nullptr /* the merge kernel */, nullptr, nullptr,
                   (unsigned*)(base + o_cnt), (LmPart*)(base + o_lm), part_bytes, ml_bytes, batch};
  std::vector<int> seqs(seq_ids, seq_ids + batch), grow(batch, 1);
  st = check_growth(m, kv, seqs, grow);
  if (st != LASER_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  Plan* p = m->static_plan;
  st = flush_pending(kv, m, s, p);
  if (st != LASER_OK) return st;
  {
    TimingScope scope(m);
    HIP_TRY(launch_fill_u32(sc.attn_cnt, (int)cnt_n, 0u, s));  // the array keeps the last call's contents
    HIP_TRY(launch_fill_u32(sc.kcnt, (int)(kcnt_bytes / 4), 0u, s));
  }
  p->M = batch;
  p->n_out = batch;
  p->n_bt = 0;
  std::vector<PageUpdate> upd;
  for (int b = 0; b < batch; ++b) {
    const int pos = kv->pool.len(seqs[b]);
    kv->pool.append(seqs[b], 1, &upd);
    p->rows[b] = RowDesc{seqs[b], pos, 0, b};
    p->outs[b] = OutDesc{b, 0, b, 0};
  }
  push_updates(*p, upd);
  PlanIO io{};
  io.tok_src[0] = io.tok_src[1] = d_tokens;
  io.tok_dst[0] = d_next;
  io.p_dst[0] = d_max_prob;
  io.logits[0] = d_logits;
  return run_forward(m, kv, *p, io, s, /*allow_graph=*/false, &sc);
}

extern "C" laser_status laser_prefill(laser_model* m, laser_kv* kv, int seq_id, const int32_t* d_tokens, int n,
                                      float* d_logits_last, void* stream) {
  laser_status st = check_ready(m, kv);
  if (st != LASER_OK) return st;
  if (!d_tokens || n < 1) return laser_fail(LASER_ERR_INVALID_ARG, "need n >= 1 tokens");
  std::vector<int> seqs{seq_id}, grow{n};
  st = check_growth(m, kv, seqs, grow);
  if (st != LASER_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  st = flush_pending(kv, m, s);
  if (st != LASER_OK) return st;
  Plan* p = new (std::nothrow) Plan;
  if (!p) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  for (int c0 = 0; c0 < n && st == LASER_OK; c0 += m->max_rows) {
    const int M = std::min(m->max_rows, n - c0);
    p->M = M;
    p->n_bt = 0;
    std::vector<PageUpdate> upd;
    const int pos0 = kv->pool.len(seq_id);
    kv->pool.append(seq_id, M, &upd);
    for (int i = 0; i < M; ++i) p->rows[i] = RowDesc{seq_id, pos0 + i, 0, c0 + i};
    push_updates(*p, upd);
    const bool last = c0 + M >= n;
    p->n_out = (last && d_logits_last) ? 1 : 0;
    p->outs[0] = OutDesc{M - 1, 0, 0, 0};
    PlanIO io{};
    io.tok_src[0] = io.tok_src[1] = d_tokens;
    io.tok_dst[0] = m->wsp<int>(m->lay.tok_buf);
    io.p_dst[0] = m->wsp<float>(m->lay.p_buf);
    io.logits[0] = d_logits_last;
    st = run_forward(m, kv, *p, io, s, /*allow_graph=*/false);  // one-off chunk shapes
  }
  delete p;
  return st;
}

// Trial-token forwards j = 1..T-1 of a probe: row r feeds t_j (d_argmax[r*T + j-1]).
static laser_status run_trials(laser_model* m, laser_kv* kv, Plan* p, const std::vector<int>& seqs,
                               const std::vector<int>& base_pos, int S, int T, int32_t* d_argmax, float* probe_p,
                               float* d_logits, hipStream_t s) {
  for (int j = 1; j < T; ++j) {
    const int n = (int)seqs.size();
    p->M = n;
    p->n_out = n;
    p->n_bt = 0;
    for (int r = 0; r < n; ++r) {
      p->rows[r] = RowDesc{seqs[r], base_pos[r] + S + j - 1, 0, r * T + j - 1};
      p->outs[r] = OutDesc{r, 0, r * T + j, 0};
    }
    PlanIO io{};
    io.tok_src[0] = io.tok_src[1] = d_argmax;
    io.tok_dst[0] = d_argmax;
    io.p_dst[0] = probe_p;
    io.logits[0] = d_logits;
    laser_status st = run_forward(m, kv, *p, io, s);
    if (st != LASER_OK) return st;
  }
  return LASER_OK;
}

extern "C" laser_status laser_probe_confidence(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                                               const int32_t* d_suffix, int S, int T, float* d_conf, int32_t* d_argmax,
                                               float* d_logits, void* stream) {
  laser_status st = check_ready(m, kv);
  if (st != LASER_OK) return st;
  if (!seq_ids || !d_suffix || !d_conf || !d_argmax) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (S < 1 || T < 1 || T > kMaxT) return laser_fail(LASER_ERR_INVALID_ARG, "need S >= 1 and 1 <= T <= %d", kMaxT);
  if (batch < 1 || (long long)batch * S > m->max_rows)
    return laser_fail(LASER_ERR_INVALID_ARG, "batch*S must be in [1, %d]", m->max_rows);
  std::vector<int> seqs(seq_ids, seq_ids + batch), grow(batch, S + T - 1);
  st = check_growth(m, kv, seqs, grow);
  if (st != LASER_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  st = flush_pending(kv, m, s);
  if (st != LASER_OK) return st;
  Plan* p = new (std::nothrow) Plan;
  if (!p) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  std::vector<int> L0(batch);
  std::vector<PageUpdate> upd;
  for (int r = 0; r < batch; ++r) {
    L0[r] = kv->pool.len(seqs[r]);
    kv->pool.append(seqs[r], S + T - 1, &upd);  // scratch positions for the suffix and fed-back trials
  }
  float* probe_p = m->wsp<float>(m->lay.probe_p);
  // chunk forward: the S suffix rows of every request; the last row of each gives t_1, p_1
  p->M = batch * S;
  p->n_out = batch;
  p->n_bt = 0;
  push_updates(*p, upd);
  for (int r = 0; r < batch; ++r) {
    for (int i = 0; i < S; ++i) p->rows[r * S + i] = RowDesc{seqs[r], L0[r] + i, 0, i};
    p->outs[r] = OutDesc{r * S + S - 1, 0, r * T, 0};
  }
  PlanIO io{};
  io.tok_src[0] = io.tok_src[1] = d_suffix;
  io.tok_dst[0] = d_argmax;
  io.p_dst[0] = probe_p;
  io.logits[0] = d_logits;
  st = run_forward(m, kv, *p, io, s);
  if (st == LASER_OK) st = run_trials(m, kv, p, seqs, L0, S, T, d_argmax, probe_p, d_logits, s);
  if (st == LASER_OK) {
    TimingScope scope(m);
    hipError_t e = timed(m, LASER_K_OTHER, s, [&] { return launch_confidence(probe_p, T, batch, d_conf, s); });
    if (e != hipSuccess) st = laser_fail(LASER_ERR_HIP, "confidence: %s", hipGetErrorString(e));
  }
  for (int r = 0; r < batch; ++r) kv->pool.truncate(seqs[r], L0[r]);  // the probe leaves no trace
  delete p;
  return st;
}

extern "C" laser_status laser_step_mixed(laser_model* m, laser_kv* kv, int batch, const int32_t* seq_ids,
                                         const int32_t* d_tokens, int32_t* d_next, float* d_max_prob, int n_probe,
                                         const int32_t* probe_idx, const int32_t* d_suffix, int S, int T, float* d_conf,
                                         int32_t* d_argmax, void* stream) {
  laser_status st = check_ready(m, kv);
  if (st != LASER_OK) return st;
  if (!seq_ids || !d_tokens || !d_next || !d_max_prob) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (batch < 1 || n_probe < 0 || n_probe > batch) return laser_fail(LASER_ERR_INVALID_ARG, "bad batch / n_probe");
  if (n_probe > 0) {
    if (!probe_idx || !d_suffix || !d_conf || !d_argmax) return laser_fail(LASER_ERR_INVALID_ARG, "NULL probe argument");
    if (S < 1 || T < 1 || T > kMaxT) return laser_fail(LASER_ERR_INVALID_ARG, "need S >= 1 and 1 <= T <= %d", kMaxT);
  }
  if ((long long)batch + (long long)S * n_probe > m->max_rows)
    return laser_fail(LASER_ERR_INVALID_ARG, "batch + S*n_probe exceeds max_rows %d", m->max_rows);
  std::vector<int> probing(batch, -1);
  for (int i = 0; i < n_probe; ++i) {
    const int b = probe_idx[i];
    if (b < 0 || b >= batch || probing[b] >= 0) return laser_fail(LASER_ERR_INVALID_ARG, "bad or repeated probe_idx");
    if (i > 0 && b <= probe_idx[i - 1]) return laser_fail(LASER_ERR_INVALID_ARG, "probe_idx must be increasing");
    probing[b] = i;
  }
  std::vector<int> seqs(seq_ids, seq_ids + batch), grow(batch, 1);
  for (int b = 0; b < batch; ++b)
    if (probing[b] >= 0) grow[b] += S + T - 1;
  st = check_growth(m, kv, seqs, grow);
  if (st != LASER_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  st = flush_pending(kv, m, s);
  if (st != LASER_OK) return st;
  Plan* p = new (std::nothrow) Plan;
  if (!p) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  std::vector<PageUpdate> upd;
  std::vector<int> pseqs, pbase;
  int M = 0, nout = 0;
  p->n_bt = 0;
  // committed decode positions first (batch order), then the probes' scratch positions
  std::vector<int> pos0(batch);
  for (int b = 0; b < batch; ++b) {
    pos0[b] = kv->pool.len(seqs[b]);
    kv->pool.append(seqs[b], 1, &upd);
  }
  for (int b = 0; b < batch; ++b)
    if (probing[b] >= 0) kv->pool.append(seqs[b], S + T - 1, &upd);
  for (int b = 0; b < batch; ++b) {
    const int pos = pos0[b];
    p->rows[M] = RowDesc{seqs[b], pos, 0, b};
    p->outs[nout++] = OutDesc{M, 0, b, 0};
    ++M;
    if (probing[b] >= 0) {
      const int i = probing[b];
      for (int q = 0; q < S; ++q) p->rows[M + q] = RowDesc{seqs[b], pos + 1 + q, 1, q};
      p->outs[nout++] = OutDesc{M + S - 1, 1, i * T, 0};
      M += S;
      pseqs.push_back(seqs[b]);
      pbase.push_back(pos + 1);
    }
  }
  p->M = M;
  p->n_out = nout;
  push_updates(*p, upd);
  float* probe_p = m->wsp<float>(m->lay.probe_p);
  PlanIO io{};
  io.tok_src[0] = d_tokens;
  io.tok_src[1] = d_suffix;
  io.tok_dst[0] = d_next;
  io.p_dst[0] = d_max_prob;
  io.tok_dst[1] = d_argmax;
  io.p_dst[1] = probe_p;
  st = run_forward(m, kv, *p, io, s);
  if (st == LASER_OK && n_probe > 0) st = run_trials(m, kv, p, pseqs, pbase, S, T, d_argmax, probe_p, nullptr, s);
  if (st == LASER_OK && n_probe > 0) {
    TimingScope scope(m);
    hipError_t e = timed(m, LASER_K_OTHER, s, [&] { return launch_confidence(probe_p, T, n_probe, d_conf, s); });
    if (e != hipSuccess) st = laser_fail(LASER_ERR_HIP, "confidence: %s", hipGetErrorString(e));
  }
  for (size_t i = 0; i < pseqs.size(); ++i) kv->pool.truncate(pseqs[i], pbase[i]);
  delete p;
  return st;
}

// ----------------------------------------------------------------------------- forks, spans

extern "C" laser_status laser_kv_fork(laser_kv* kv, int src_seq, int dst_seq, void* stream) {
  if (!kv_of(kv)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed kv");
  laser_model* m = const_cast<laser_model*>(kv->m);
  if (!model_of(m) || !m->finalized) return laser_fail(LASER_ERR_STATE, "model not finalized");
  PageCopy c{};
  bool has = false;
  std::vector<PageUpdate> upd;
  const int st = kv->pool.fork(src_seq, dst_seq, &upd, &c, &has);
  if (st != LASER_OK) return (laser_status)st;
  kv->pending.insert(kv->pending.end(), upd.begin(), upd.end());  // block-table rows travel with the next plan
  if (has) {
    hipStream_t s = (hipStream_t)stream;
    const laser_model_desc& d = m->desc;
    TimingScope scope(m);
    const hipError_t e = timed(m, LASER_K_OTHER, s, [&] {
      return launch_page_copy(m->kv_es, kv->kpool, kv->vpool, kv->pool.num_pages(), d.n_layers,
                              d.n_kv_heads, d.head_dim, c.src, c.dst, s);
    });
    if (e != hipSuccess) return laser_fail(LASER_ERR_HIP, "page copy: %s", hipGetErrorString(e));
  }
  return LASER_OK;
}

extern "C" laser_status laser_forward(laser_model* m, laser_kv* kv, int n_spans, const laser_span* spans,
                                      const int32_t* d_tok0, const int32_t* d_tok1, int32_t* d_out_tok0, float* d_out_p0,
                                      int32_t* d_out_tok1, float* d_out_p1, float* d_out_logits0,
                                      float* d_out_logits1, void* stream) {
  laser_status st = check_ready(m, kv);
  if (st != LASER_OK) return st;
  if (n_spans < 1 || !spans) return laser_fail(LASER_ERR_INVALID_ARG, "need at least one span");
  long long rows = 0;
  std::vector<int> seqs, grow;
  for (int i = 0; i < n_spans; ++i) {
    const laser_span& sp = spans[i];
    if (sp.n_tokens < 1 || sp.tok_off < 0 || (sp.tok_sel != 0 && sp.tok_sel != 1))
      return laser_fail(LASER_ERR_INVALID_ARG, "span %d: bad n_tokens, tok_sel or tok_off", i);
    if (!(sp.tok_sel ? d_tok1 : d_tok0)) return laser_fail(LASER_ERR_INVALID_ARG, "span %d: its token array is NULL", i);
    if (sp.out) {
      if ((sp.out_sel != 0 && sp.out_sel != 1) || sp.out_off < 0)
        return laser_fail(LASER_ERR_INVALID_ARG, "span %d: bad out_sel or out_off", i);
      if (!(sp.out_sel ? d_out_tok1 : d_out_tok0) || !(sp.out_sel ? d_out_p1 : d_out_p0))
        return laser_fail(LASER_ERR_INVALID_ARG, "span %d: its output arrays are NULL", i);
    }
    rows += sp.n_tokens;
    seqs.push_back(sp.seq);
    grow.push_back(sp.n_tokens);
  }
  if (rows > m->max_rows) return laser_fail(LASER_ERR_INVALID_ARG, "%lld rows exceed max_rows %d", rows, m->max_rows);
  st = check_growth(m, kv, seqs, grow);
  if (st != LASER_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  st = flush_pending(kv, m, s);
  if (st != LASER_OK) return st;
  Plan* p = new (std::nothrow) Plan;
  if (!p) return laser_fail(LASER_ERR_INVALID_ARG, "allocation failed");
  p->M = 0;
  p->n_out = 0;
  p->n_bt = 0;
  std::vector<PageUpdate> upd;
  for (int i = 0; i < n_spans; ++i) {
    const laser_span& sp = spans[i];
    const int pos0 = kv->pool.len(sp.seq);
    kv->pool.append(sp.seq, sp.n_tokens, &upd);
    for (int t = 0; t < sp.n_tokens; ++t) p->rows[p->M + t] = RowDesc{sp.seq, pos0 + t, sp.tok_sel, sp.tok_off + t};
    p->M += sp.n_tokens;
    if (sp.out) p->outs[p->n_out++] = OutDesc{p->M - 1, sp.out_sel, sp.out_off, 0};
  }
  push_updates(*p, upd);
  PlanIO io{};
  io.tok_src[0] = d_tok0;
  io.tok_src[1] = d_tok1;
  io.tok_dst[0] = d_out_tok0;
  io.tok_dst[1] = d_out_tok1;
  io.p_dst[0] = d_out_p0;
  io.p_dst[1] = d_out_p1;
  io.logits[0] = d_out_logits0;
  io.logits[1] = d_out_logits1;
  st = run_forward(m, kv, *p, io, s);
  delete p;
  return st;
}

extern "C" laser_status laser_confidence(laser_model* m, const float* d_p, int T, int n, float* d_conf, void* stream) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!d_p || !d_conf || T < 1 || n < 1) return laser_fail(LASER_ERR_INVALID_ARG, "bad argument");
  hipStream_t s = (hipStream_t)stream;
  TimingScope scope(m);
  const hipError_t e = timed(m, LASER_K_OTHER, s, [&] { return launch_confidence(d_p, T, n, d_conf, s); });
  if (e != hipSuccess) return laser_fail(LASER_ERR_HIP, "confidence: %s", hipGetErrorString(e));
  return LASER_OK;
}

// ----------------------------------------------------------------------------- ATP cues

extern "C" laser_status laser_atp_bitmap(const int32_t* ids, int n_ids, int vocab, uint32_t* words_out) {
  if (!words_out || n_ids < 0 || vocab < 1 || (n_ids > 0 && !ids)) return laser_fail(LASER_ERR_INVALID_ARG, "bad argument");
  for (int i = 0; i < n_ids; ++i)
    if (ids[i] < 0 || ids[i] >= vocab) return laser_fail(LASER_ERR_INVALID_ARG, "id %d outside the vocabulary", ids[i]);
  const int nw = (vocab + 31) / 32;
  for (int w = 0; w < nw; ++w) words_out[w] = 0u;
  for (int i = 0; i < n_ids; ++i) words_out[ids[i] >> 5] |= 1u << (ids[i] & 31);
  return LASER_OK;
}

extern "C" laser_status laser_atp_match(const int32_t* d_tokens, int n, const uint32_t* d_bitmap, int vocab,
                                        int32_t* d_flags, void* stream) {
  if (!d_tokens || !d_bitmap || !d_flags || n < 1 || vocab < 1) return laser_fail(LASER_ERR_INVALID_ARG, "bad argument");
  const hipError_t e = launch_atp_match(d_tokens, n, d_bitmap, vocab, d_flags, (hipStream_t)stream);
  if (e != hipSuccess) return laser_fail(LASER_ERR_HIP, "atp match: %s", hipGetErrorString(e));
  return LASER_OK;
}

// ----------------------------------------------------------------------------- graphs

extern "C" laser_status laser_model_set_graphs(laser_model* m, int enable) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  m->use_graphs = enable != 0;
  return LASER_OK;
}

extern "C" laser_status laser_model_graph_stats(const laser_model* m, long long* captures, int* cached) {
  if (!model_of(const_cast<laser_model*>(m))) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (!captures || !cached) return laser_fail(LASER_ERR_INVALID_ARG, "null output pointer");
  *captures = m->graph_captures;
  *cached = (int)m->graphs.size();
  return LASER_OK;
}

extern "C" laser_status laser_model_set_attn_merge(laser_model* m, int fused, int max_splits) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if ((fused != 0 && fused != 1) || max_splits < 2 || max_splits > kAttnMaxWG)
    return laser_fail(LASER_ERR_INVALID_ARG, "fused must be 0 or 1 and max_splits in [2, %d]", kAttnMaxWG);
  m->attn_fuse = fused;
  m->attn_fuse_max = max_splits;
  return LASER_OK;
}

extern "C" laser_status laser_model_set_oproj_merge(laser_model* m, int mode) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (mode < 0 || mode > 2) return laser_fail(LASER_ERR_INVALID_ARG, "mode must be 0, 1 or 2");
  m->oproj_merge = mode;  // (captured forwards are keyed on where the merge runs)
  return LASER_OK;
}

extern "C" laser_status laser_model_set_gemm_kernel(laser_model* m, int mode) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (mode < 0 || mode > 2) return laser_fail(LASER_ERR_INVALID_ARG, "gemm kernel mode must be 0, 1 or 2");
  if (mode != m->gemm_kernel) drop_graphs(m);  // captured forwards hold the previous choice
  m->gemm_kernel = mode;
  return LASER_OK;
}

// ----------------------------------------------------------------------------- timing

// Restarts the event pool once no class holds unread spans (after its last event is done).
static laser_status maybe_reset_pool(laser_model* m) {
  for (const auto& t : m->timers)
    if (!t.spans.empty()) return LASER_OK;
  if (m->ev_used > 0) HIP_TRY(hipEventSynchronize(m->ev_pool[m->ev_used - 1]));
  m->ev_used = 0;
  m->last_stop = -1;
  return LASER_OK;
}

extern "C" laser_status laser_timing_enable(laser_model* m, int kernel_class, int enable) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (kernel_class < 0 || kernel_class >= LASER_K_NCLASS) return laser_fail(LASER_ERR_INVALID_ARG, "bad kernel class");
  m->timers[kernel_class].enabled = enable != 0;
  m->timers[kernel_class].spans.clear();
  return maybe_reset_pool(m);
}

extern "C" laser_status laser_timing_read(laser_model* m, int kernel_class, double* total_ms, int* launches) {
  if (!model_of(m)) return laser_fail(LASER_ERR_STATE, "invalid or destroyed model");
  if (kernel_class < 0 || kernel_class >= LASER_K_NCLASS) return laser_fail(LASER_ERR_INVALID_ARG, "bad kernel class");
  if (!total_ms || !launches) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  Timer& t = m->timers[kernel_class];
  double tot = 0.0;
  if (!t.spans.empty()) HIP_TRY(hipEventSynchronize(m->ev_pool[t.spans.back().second]));
  for (const auto& sp : t.spans) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, m->ev_pool[sp.first], m->ev_pool[sp.second]));
    tot += ms;
  }
  *total_ms = tot;
  *launches = (int)t.spans.size();
  t.spans.clear();
  return maybe_reset_pool(m);
}
