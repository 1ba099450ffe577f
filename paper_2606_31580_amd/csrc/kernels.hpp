// Internal interface between the host runtime and the gfx950 kernels of liblaser.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace laser {

constexpr int kMaxRows = 64;      // rows (tokens) of one forward
constexpr int kPage = 16;         // positions per KV page
constexpr int kMaxBt = 1024;      // block-table updates carried by one plan
constexpr int kAttnWaves = 4;     // waves per attention workgroup (one split each)
constexpr int kAttnMaxWG = 128;   // attention workgroups (page splits) per (group, kv head)
constexpr int kMaxGroups = 2 * kMaxRows;  // own groups (one per run of rows) + shared-page groups
constexpr int kMaxAttnItems = 8192;       // attention workgroups per kv head
constexpr int kGemmThreads = 256; // 4 waves
constexpr int kGemvMaxThreads = 512;
constexpr int kMfmaMaxWaves = 8;    // waves of an MFMA projection workgroup with few row groups
constexpr int kMaxKsplit = 4;       // K shares of a residual projection on the MFMA path
constexpr int kKsCntStride = 16;    // K-share arrival counters 64 bytes apart

// One row of a forward: request slot, position, and where its input token id lives.
struct RowDesc {
  int seq, pos, tok_sel, tok_off;  // token = tok_base[tok_sel][tok_off]
};
// Contiguous rows that attend over pages [pbeg, npages) of sequence seq's block table: the
// rows of one request, or (shared prefix) the rows of a request and its forks over the full
// pages they share, whose own later pages are then separate groups.
struct GroupDesc {
  int seq, row0, nrows, npages, pps, nwg;  // npages: end page; pps: pages per wave split; nwg: workgroups
  int maxpos;                              // last position any row of the group sees
  int pbeg;                                // first page
  int slot0;                               // first partial slot of the group's workgroups
  int direct;                              // the group alone covers its rows in one workgroup: no merge
  int fused;                               // one row, several workgroups: merged by the last of them
};
// One attention workgroup (per kv head): a group's 16-column query tile over 4 runs of pages,
// wave w's run [p0 + w pps, min(p0 + (w + 1) pps, pend)).  nrows == 0: padding, no work.
// A one-row group split over several workgroups may merge its splits itself ("fused"): then
// nrows carries the split count in bits 8-15 and the group's arrival counter in bits 16-23,
// and the last workgroup of the group to finish combines every split's partial.
struct AttnItem {
  int seq, row0, nrows;  // the group's block table and rows (bits 0-7; fused: see above)
  int p0, pend, pps;
  int maxpos;            // last position any row of the group sees
  int info;              // tile (bits 0-7) | partial slot (bits 8-23) | direct output (bit 24)
};
constexpr int kAttnCntStride = 16;  // arrival counters 64 bytes apart: [kv head][group]
// LM-head output row: activation row, destination (sel, off) for token / prob / logits.
struct OutDesc {
  int row, sel, off, pad;
};
struct BtUpdate {
  int seq, idx, page;
};

// Caller buffers of one forward (they may change from call to call, so they travel in the
// plan rather than in kernel arguments, which a replayed graph keeps fixed).
struct PlanIO {
  const int* tok_src[2];  // input token of row r: tok_src[rows[r].tok_sel][rows[r].tok_off]
  int* tok_dst[2];        // greedy token of output o: tok_dst[outs[o].sel][outs[o].off]
  float* p_dst[2];        // its max-softmax probability, same index
  float* logits[2];       // optional logits rows [..][vocab], same index; may be null
};

// Everything the kernels of one forward need that changes per call; uploaded once (the used
// part of each array).
struct alignas(16) Plan {  // (16-byte aligned arrays: k_plan_fetch copies 16-byte chunks)
  int M, n_groups, n_out, n_bt, n_items;
  // split merge carried by the O-projection's launch: the value every layer's merge counter
  // reaches once this forward's merge workgroups of that layer have stored their outputs
  unsigned merge_target;
  PlanIO io;
  RowDesc rows[kMaxRows];
  int row_nslots[kMaxRows];  // attention partial slots of each row (over all its groups)
  OutDesc outs[kMaxRows];
  alignas(16) AttnItem items[kMaxAttnItems];
  alignas(16) BtUpdate bt[kMaxBt];
  GroupDesc groups[kMaxGroups];  // (host side: the kernels read the work items)
};

// Softmax statistics of one group of vocabulary rows for one output row.
struct LmPart {
  float mx, sum;
  int idx, pad;
};

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LMHEAD = 3 };

// Output rows per workgroup of a projection on the MFMA path (one matrix-core tile).  The
// VALU path takes 8, or 6 / 7 where that spreads the groups evenly over the compute units
// (launch_gemm's rw).  Rotary and gate/up rows come in pairs, half of a group each.
constexpr int rows_per_group(int, bool) { return 16; }

struct GemmArgs {
  // weights (row-major [rows][K] in the model dtype)
  const void* w0;
  const void* w1;
  const void* w2;
  int K, N, M, n_groups;
  int nr;   // MFMA path: row groups per workgroup (1, 2, or 4 at 2-3 activation tiles)
  int nrw;  // MFMA path: 0, or row groups per wave of the row-wave kernel (1, 2; 4 waves)
  int gv_threads, gv_u;  // VALU path: threads per workgroup and chunks in flight per thread (0: defaults)
  // MFMA path: the weights in tile order (null: read the row-major tensors).  Group g, step s
  // (32 columns) is a block of 64 lanes x 16 bytes (x 2 for fp32) at (g * tsteps + s) blocks.
  const char* wtile;
  int tsteps;
  // A operand: fp32 activation rows [row][ldx]; optional RMSNorm over the full row (gain)
  const float* x;
  int ldx;
  const void* gain;
  float eps;
  int row_map;  // A row m = plan->outs[m].row (LM head)
  const Plan* plan;
  // EPI_QKV
  const void* b0;
  const void* b1;
  const void* b2;
  int hq, hkv, hd;
  const float2* rope;  // [max_positions][hd/2] (cos, sin)
  float* q_out;        // [M][hq][hd]
  void* kpool;
  void* vpool;
  const int* bt;
  int max_pps, num_pages, layer;
  int kv_fp8;  // K/V stored as E4M3 (else in the weight type)
  // EPI_RESID
  float* h;  // [M][N]
  // MFMA path, EPI_RESID only: K split across `ksplit` workgroups per row group (1: none).
  // Each writes its partial outputs to kpart[ks][M][N].  With kcnt (one counter per block of
  // row groups, kKsCntStride apart, zero between kernels) each counts its arrival and the last
  // to arrive adds the shares, in share order, to h and re-arms the counter; without it,
  // launch_ksplit_reduce adds them.
  int ksplit;
  float* kpart;
  unsigned* kcnt;
  // EPI_SWIGLU
  float* act;  // [M][F]
  int F;
  // EPI_LMHEAD (logits destinations come from plan->io)
  LmPart* lm_part;  // [M][n_groups]
};

struct AttnArgs {
  const Plan* plan;
  const float* q;  // [M][hq][hd]
  float* o;        // [M][hq][hd]
  const void* kpool;
  const void* vpool;
  const int* bt;
  int max_pps, num_pages, layer;
  int hq, hkv, G, max_rows;
  float scale_log2;
  float* part;  // [hkv][kAttnMaxWG][max_rows*G][hd]
  float* ml;    // [hkv][kAttnMaxWG][max_rows*G][2]
  uint32_t part_bytes, ml_bytes;
  unsigned* cnt;  // fused groups' arrival counters [hkv][kMaxGroups] x kAttnCntStride; zero between kernels
};

// Kernel timing hooks.  `start`/`stop` are bound to the next launch only; when `next_stop`
// is set (a timing session), every launch without an explicit stop event gets one from it,
// so the end of each kernel is known.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  hipEvent_t (*next_stop)(void*) = nullptr;
  void* ctx = nullptr;
};
LaunchEvents& launch_events();

template <class K, class... Args>
inline hipError_t launch_k(K kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
  LaunchEvents& e = launch_events();
  hipEvent_t stop = e.stop;
  if (!stop && e.next_stop) stop = e.next_stop(e.ctx);
  if (e.start || stop)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e.start, stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
  e.start = e.stop = nullptr;
  return hipGetLastError();
}

// dtype: 0 fp32, 1 bf16.  mode: 1..4 VALU rows per forward, 5..8 MFMA with 1..4 m-tiles.
// rw: rows per workgroup (VALU: QKV 6 or 8, residual 6, 7 or 8, others 8; MFMA: 16).
hipError_t launch_gemm(int dtype, int mode, int epi, int rw, const GemmArgs& a, hipStream_t s);
hipError_t launch_ksplit_reduce(const GemmArgs& a, hipStream_t s);

// The attention split merge carried by the first workgroups of the O-projection's launch
// (VALU path, 1-2 rows): merge workgroup b < nwg combines the partials of (row b / hq, head
// b % hq) like k_attn_merge, stores o with device-scope stores and bumps the layer's counter;
// the projection's workgroups issue their weight loads, wait (bounded) until the counter
// reaches plan->merge_target, then read o with device-scope loads.  The counter only grows:
// each forward adds nwg per layer and the host carries the running total in the plan.  The
// counter has kMgReplicas copies (kKsCntStride apart), each merge workgroup bumps all of them
// and projection workgroup g polls copy g mod kMgReplicas (7B shape, 512 projection
// workgroups: the projection with the merge took 13.1-13.4 us with one copy, 11.5 us with 16).
constexpr int kMgReplicas = 64;
struct MergeArgs {
  const float* part;  // attention partials [hkv][kAttnMaxWG][max_rows * G][hd]
  const float* ml;    // their (m, l) pairs, same index
  unsigned* cnt;      // this layer's counter replicas
  uint32_t o_bytes;   // bytes of o (the projection's activation rows, GemmArgs::x)
  int hq, G, hd, max_rows, nslots, nwg;  // nslots: bound on every row's slot count; nwg = M * hq
};
hipError_t launch_gemv_merged(int dtype, int rw, const GemmArgs& a, const MergeArgs& mg, hipStream_t s);
// QKV of a wide forward (bf16 weights; a.M of 33 to 64 rows) over K slices of kQSliceSteps
// 32-column steps, kQSliceGroups row groups per workgroup: partial sums per slice in qpart
// [ceil(K / (32 kQSliceSteps))][M][N], the rows' sums of squares per slice in sqpart [slices][M],
// then the summing / norm / epilogue kernel.
constexpr int kQSliceSteps = 16, kQSliceGroups = 16;
hipError_t launch_qkv_slices(const GemmArgs& a, float* qpart, float* sqpart, hipStream_t s);
// Writes the tile-order copy of one projection's weights (the MFMA path's 16-row groups of
// `a`, as weight_row maps them) to dst: a.n_groups groups x ceil(K/32) steps.
hipError_t launch_tile_weights(int dtype, int epi, const GemmArgs& a, char* dst, hipStream_t s);
// dtype: the KV element type, 0 fp32, 1 bf16, 2 fp8 (E4M3).
hipError_t launch_attn(int dtype, int hd, const AttnArgs& a, dim3 grid, hipStream_t s);
hipError_t launch_attn_merge(const AttnArgs& a, int M, int hd, int nslots, hipStream_t s);  // nslots >= every group's nwg
hipError_t launch_lm_reduce(const Plan* plan, const LmPart* part, int n_groups, int n_out, hipStream_t s);
hipError_t launch_embed(int dtype, const Plan* plan, int M, const void* embed, int d, int vocab, float* h, int* bt,
                        int max_pps, hipStream_t s);
hipError_t launch_apply_bt(const Plan* plan, int* bt, int max_pps, hipStream_t s);
// Copies a staged plan (pinned host slot) to the device plan slot; the kernel's address, so a
// captured forward's copy can be pointed at the next slot before each replay.
hipError_t launch_plan_fetch(const Plan* src, Plan* dst, hipStream_t s);
const void* plan_fetch_kernel();
// kv_es: bytes per KV element (1 fp8, 2 bf16, 4 fp32); the copy moves raw elements.
hipError_t launch_kv_copy(int kv_es, int to_pool, void* kpool, void* vpool, const int* bt, int max_pps,
                          int num_pages, int n_layers, int hkv, int hd, int seq, int len, void* k_lin,
                          void* v_lin, hipStream_t s);
hipError_t launch_confidence(const float* p, int T, int n, float* conf, hipStream_t s);
hipError_t launch_fill_u32(unsigned* p, int n, unsigned v, hipStream_t s);
hipError_t launch_atp_match(const int* tokens, int n, const unsigned* bitmap, int vocab, int* flags, hipStream_t s);
hipError_t launch_page_copy(int kv_es, void* kpool, void* vpool, int num_pages, int n_layers, int hkv, int hd, int src,
                            int dst, hipStream_t s);

}  // namespace laser
