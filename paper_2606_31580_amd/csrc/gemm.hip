// Weight-streaming projections of the decoder (the bulk of every decode step's HBM bytes).
//
// One kernel family computes Y = A W^T for A = M activation rows (fp32) and a row-major
// weight matrix W [rows][K] (bf16 or fp32), fused with what precedes and follows it:
//   RMSNorm   applied as a per-row scale after the product: W (h * rms * g) = rms W (h * g),
//             with sum(h^2) accumulated from the same activation chunks the main loop reads;
//   epilogue  EPI_QKV    bias, rotary embedding of q/k, K/V appended to the paged cache;
//             EPI_RESID  residual add into h;
//             EPI_SWIGLU silu(gate) * up;
//             EPI_LMHEAD logits and per-group (max, sum exp, argmax) for k_lm_reduce,
//                        stored [row][group].
// A workgroup owns complete output rows (6-8 on the VALU path, 1, 2 or 4 groups of 16 on the
// MFMA path), so every epilogue stays inside the workgroup: its waves split K and are
// reduced through LDS in a fixed order, with no synchronisation between workgroups and
// results that do not depend on scheduling.  The one exception is the MFMA path's residual
// projections, which may split K over 2-4 workgroups: each writes its partial rows, and the
// shares are added to h in share order: by the last of the workgroups to arrive (an atomic
// counter) at 2 shares, else by k_ksplit_reduce (ksplit_finish).
// Main loops:
//   VALU (decode: 1-4 rows; the runtime uses it up to 2): each thread streams 16-byte
//       non-temporal loads of the group's rows, two chunks at a time (a wave instruction
//       reads 1 KB contiguous of one row).
//   MFMA (more rows: batches, probe chunks, prefill) 16x16x32 bf16: weights are the B
//       operand (optionally read from the tile-order copy), activations the A operand split
//       into bf16 hi + lo so the product keeps ~16 significand bits of fp32 activations;
//       fp32 weights are split too.  One activation fragment feeds every row group of the
//       workgroup.
#include <type_traits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace laser {

// One of three kernel-argument pointers chosen by flags, formed arithmetically: a select
// between argument loads would be folded into a load at a selected argument offset, which
// forces the whole argument block into scratch memory.
__device__ __forceinline__ const void* pick3(bool c0, bool c1, const void* p0, const void* p1, const void* p2) {
  const uint64_t u0 = (uint64_t)p0, u1 = (uint64_t)p1, u2 = (uint64_t)p2;
  const uint64_t f0 = c0, f1 = !c0 && c1, f2 = !c0 && !c1;
  return (const void*)(u0 * f0 + u1 * f1 + u2 * f2);
}

template <class T>
__device__ __forceinline__ T* pick2(bool c0, T* p0, T* p1) {
  const uint64_t u0 = (uint64_t)p0, u1 = (uint64_t)p1;
  return (T*)(u0 * (uint64_t)c0 + u1 * (uint64_t)(!c0));
}

// Rotary pair gp of the QKV rows: pair (i, i + hd/2) of head h, heads numbered q, then k,
// then v.  A workgroup holds RW/2 consecutive pairs (they may span two heads).
struct QkvPair {
  int hh, i;  // head within q, k or v; pair index within the head
  bool isq, isk;
  const void* bias;
  const void* w;
};

__device__ __forceinline__ QkvPair qkv_pair(const GemmArgs& a, int gp) {
  QkvPair q;
  const int half = a.hd >> 1;
  const int h = gp / half;
  q.i = gp - h * half;
  q.isq = h < a.hq;
  q.isk = !q.isq && h < a.hq + a.hkv;
  q.hh = q.isq ? h : (q.isk ? h - a.hq : h - a.hq - a.hkv);
  q.bias = pick3(q.isq, q.isk, a.b0, a.b1, a.b2);
  q.w = pick3(q.isq, q.isk, a.w0, a.w1, a.w2);
  return q;
}

// Row j (< RW) of workgroup g: its weights.  QKV groups hold RW/2 rotary pairs, SwiGLU
// groups RW/2 gate rows and the matching up rows; rows past the matrix read row 0 (their
// results are discarded).
template <class WT, int EPI, int RW>
__device__ __forceinline__ const char* weight_row(const GemmArgs& a, int g, int j) {
  constexpr int P = RW / 2;
  const size_t rowbytes = (size_t)a.K * sizeof(WT);
  if (EPI == EPI_QKV) {
    const int jj = j < P ? j : j - P;
    int gp = P * g + jj;
    if (gp >= (a.hq + 2 * a.hkv) * (a.hd >> 1)) gp = 0;
    const QkvPair q = qkv_pair(a, gp);
    const int dim = j < P ? q.i : (a.hd >> 1) + q.i;
    return (const char*)q.w + (size_t)(q.hh * a.hd + dim) * rowbytes;
  } else if (EPI == EPI_SWIGLU) {
    int r = P * g + (j % P);
    if (r >= a.F) r = 0;
    return (const char*)pick3(j < P, true, a.w0, a.w1, a.w1) + (size_t)r * rowbytes;
  } else {
    int r = RW * g + j;
    if (r >= a.N) r = 0;
    return (const char*)a.w0 + (size_t)r * rowbytes;
  }
}

__device__ __forceinline__ int a_src_row(const GemmArgs& a, int m) { return a.row_map ? a.plan->outs[m].row : m; }

// Sum over the 64 lanes of NV values at once (NV in {4, 8, 16}): each halving stage trades
// half of the values with the partner lane (32, 16, 8, then 4 lanes away; the last two
// inside a row, the 4-lane stage pairing lane i with 7 - i of its 8-lane group), then the
// lanes still holding the same value index are summed.  Returns the total of value
// idx(lane), where idx = sum over stages st of bit (5 - st) of lane times NV >> (st + 1).
template <int NV>
__device__ __forceinline__ float transpose_reduce(float* v, int lane) {
  static_assert(NV == 4 || NV == 8 || NV == 16, "NV");
#pragma unroll
  for (int i = 0; i < NV / 2; ++i) {  // 32 lanes away: lower lanes keep v[i], upper v[i + NV/2]
    float x = v[i], y = v[i + NV / 2];
    swap32(x, y);
    v[i] = x + y;
  }
#pragma unroll
  for (int i = 0; i < NV / 4; ++i) {  // 16 lanes away
    float x = v[i], y = v[i + NV / 4];
    swap16(x, y);
    v[i] = x + y;
  }
  if (NV >= 8) {  // 8 lanes away (within the row)
    const bool up = (lane & 8) != 0;
#pragma unroll
    for (int i = 0; i < NV / 8; ++i) {
      const float send = up ? v[i] : v[i + NV / 8];
      const float keep = up ? v[i + NV / 8] : v[i];
      v[i] = keep + dpp_f<kDppRowRor8>(send);
    }
  }
  if (NV >= 16) {  // the other half of the 8-lane group (lane i with 7 - i)
    const bool up = (lane & 4) != 0;
    const float send = up ? v[0] : v[1];
    const float keep = up ? v[1] : v[0];
    v[0] = keep + dpp_f<kDppHalfMirror>(send);
  }
  float t = v[0];
  // lanes that differ only below the last stage's bit hold the same index: sum them
  t += dpp_f<kDppQuad1032>(t);
  t += dpp_f<kDppQuad2301>(t);
  if (NV <= 8) t += dpp_f<kDppHalfMirror>(t);
  if (NV <= 4) t += dpp_f<kDppRowRor8>(t);
  return t;
}

template <int NV>
__device__ __forceinline__ int transpose_index(int lane) {
  int idx = 0;
#pragma unroll
  for (int st = 0; (NV >> st) > 1; ++st) idx += ((lane >> (5 - st)) & 1) * ((NV >> st) >> 1);
  return idx;
}

// ----------------------------------------------------------------------------- epilogues

// One output item of the QKV (a rotary pair of one row) or residual (one element) epilogue,
// with the global values it needs.  The VALU path fetches them while its weight loads are
// in flight, so nothing but stores is left after the reduction.
struct EpiItem {
  bool live = false;
  int m = 0, j = 0;          // activation row; pair (QKV) or row (residual) within the group
  // QKV: bias of the pair's two dims as stored (bf16 bits or fp32 bits, decoded when
  // applied, so no wait is forced at fetch time); residual: current h in v0
  uint32_t b0 = 0u, b1 = 0u;
  float v0 = 0.f;
  int pos = 0, seq = 0;      // QKV: the row's position and request
  float2 cs = {1.f, 0.f};    // QKV: cos/sin of the pair's rotation at pos
  int page = 0;              // QKV: KV page that holds pos
};

// First fetch: what depends only on the item (row descriptor, bias, current h).  Every
// load is unconditional, on a clamped index (items past the end read item 0's inputs and
// stay dead): a load inside a branch makes the compiler wait for all earlier loads, the
// weight stream included, where the branches meet.
template <class WT, int EPI, int RW>
__device__ __forceinline__ void epi_fetch_a(const GemmArgs& a, int g, int M, int idx, EpiItem& it) {
  constexpr int P = RW / 2;
  if (EPI == EPI_QKV) {
    const bool in = idx < M * P;
    const int ic = in ? idx : 0;
    it.m = ic / P;
    it.j = ic - it.m * P;
    const int gp = P * g + it.j;
    it.live = in && gp < (a.hq + 2 * a.hkv) * (a.hd >> 1);
    const QkvPair q = qkv_pair(a, it.live ? gp : 0);
    const bool has_bias = a.b0 != nullptr;  // the three biases are set together
    const char* bias = has_bias ? (const char*)q.bias : (const char*)a.plan;  // the plan: any valid address
    const size_t e0 = has_bias ? (size_t)q.hh * a.hd + q.i : 0, e1 = has_bias ? e0 + (a.hd >> 1) : 0;
    if (sizeof(WT) == 2) {
      it.b0 = ld_global<uint16_t>(bias + 2 * e0);
      it.b1 = ld_global<uint16_t>(bias + 2 * e1);
    } else {
      it.b0 = ld_global<uint32_t>(bias + 4 * e0);
      it.b1 = ld_global<uint32_t>(bias + 4 * e1);
    }
    if (!has_bias) it.b0 = it.b1 = 0u;  // +0 in either storage type
    const RowDesc rd = a.plan->rows[it.m];
    it.pos = rd.pos;
    it.seq = rd.seq;
  } else if (EPI == EPI_RESID) {
    const bool in = idx < M * RW;
    const int ic = in ? idx : 0;
    it.m = ic / RW;
    it.j = ic - it.m * RW;
    const int r = RW * g + it.j;
    it.live = in && r < a.N;
    it.v0 = a.h[(size_t)it.m * a.N + (it.live ? r : 0)];
  }
}

// Second fetch (QKV): what is addressed by the row's position (rotation, KV page), loaded
// for every item whether or not it uses it (same reason as above).
template <class WT, int EPI, int RW>
__device__ __forceinline__ void epi_fetch_b(const GemmArgs& a, int g, EpiItem& it) {
  if (EPI != EPI_QKV) return;
  constexpr int P = RW / 2;
  const QkvPair q = qkv_pair(a, it.live ? P * g + it.j : 0);
  it.cs = a.rope[(size_t)it.pos * (a.hd >> 1) + q.i];
  it.page = a.bt[(size_t)it.seq * a.max_pps + (it.pos >> 4)];
}

// Bias, rotation and stores of one item; Y holds the group's outputs [m][RW].
template <class WT, int EPI, int RW>
__device__ __forceinline__ void epi_apply(const GemmArgs& a, int g, const EpiItem& it, const float* Y) {
  if (!it.live) return;
  constexpr int P = RW / 2;
  if (EPI == EPI_QKV) {
    const QkvPair q = qkv_pair(a, P * g + it.j);
    const int dlo = q.i, dhi = (a.hd >> 1) + q.i;
    const float bias0 = sizeof(WT) == 2 ? bf2f((uint16_t)it.b0) : __uint_as_float(it.b0);
    const float bias1 = sizeof(WT) == 2 ? bf2f((uint16_t)it.b1) : __uint_as_float(it.b1);
    float ylo = Y[it.m * RW + it.j] + bias0, yhi = Y[it.m * RW + P + it.j] + bias1;
    if (q.isq || q.isk) {
      const float rlo = ylo * it.cs.x - yhi * it.cs.y;
      const float rhi = yhi * it.cs.x + ylo * it.cs.y;
      ylo = rlo;
      yhi = rhi;
    }
    if (q.isq) {
      float* qo = a.q_out + ((size_t)it.m * a.hq + q.hh) * a.hd;
      qo[dlo] = ylo;
      qo[dhi] = yhi;
    } else {
      const int t = it.pos & 15;
      const size_t blk = (((size_t)a.layer * a.num_pages + it.page) * a.hkv + q.hh) * (size_t)(16 * a.hd);
      void* pool = q.isk ? a.kpool : a.vpool;
      const size_t olo = blk + (q.isk ? k_block_off(t, dlo) : v_block_off(t, dlo));
      const size_t ohi = blk + (q.isk ? k_block_off(t, dhi) : v_block_off(t, dhi));
      if (a.kv_fp8) {
        stw<fp8_t>(pool, olo, ylo);
        stw<fp8_t>(pool, ohi, yhi);
      } else {
        stw<WT>(pool, olo, ylo);
        stw<WT>(pool, ohi, yhi);
      }
    }
  } else if (EPI == EPI_RESID) {
    a.h[(size_t)it.m * a.N + RW * g + it.j] = it.v0 + Y[it.m * RW + it.j];
  }
}

template <class WT, int RW>
__device__ __forceinline__ void epi_qkv(const GemmArgs& a, int g, int M, const float* Y) {
  for (int idx = threadIdx.x; idx < M * (RW / 2); idx += blockDim.x) {
    EpiItem it;
    epi_fetch_a<WT, EPI_QKV, RW>(a, g, M, idx, it);
    epi_fetch_b<WT, EPI_QKV, RW>(a, g, it);
    epi_apply<WT, EPI_QKV, RW>(a, g, it, Y);
  }
}

template <int RW>
__device__ __forceinline__ void epi_resid(const GemmArgs& a, int g, int M, const float* Y) {
  for (int idx = threadIdx.x; idx < M * RW; idx += blockDim.x) {
    EpiItem it;
    epi_fetch_a<float, EPI_RESID, RW>(a, g, M, idx, it);
    epi_apply<float, EPI_RESID, RW>(a, g, it, Y);
  }
}

template <int RW>
__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, int g, int M, const float* Y) {
  constexpr int P = RW / 2;
  for (int idx = threadIdx.x; idx < M * P; idx += blockDim.x) {
    const int m = idx / P, jj = idx - m * P;
    const int r = P * g + jj;
    if (r < a.F) {
      const float gt = Y[m * RW + jj], up = Y[m * RW + P + jj];
      a.act[(size_t)m * a.F + r] = gt / (1.f + expf(-gt)) * up;
    }
  }
}

template <int RW>
__device__ __forceinline__ void epi_lmhead(const GemmArgs& a, int g, int M, const float* Y) {
  const int tid = threadIdx.x;
  for (int idx = tid; idx < M * RW; idx += blockDim.x) {
    const int m = idx / RW, j = idx - m * RW;
    const int r = RW * g + j;
    const OutDesc od = a.plan->outs[m];
    float* lg = a.plan->io.logits[od.sel];
    if (r < a.N && lg != nullptr) lg[(size_t)od.off * a.N + r] = Y[idx];
  }
  if (tid < M) {
    float mx = -INFINITY;
    int arg = RW * g;  // a valid id even if no logit compares greater (NaN input)
    for (int j = 0; j < RW; ++j) {
      const int r = RW * g + j;
      if (r < a.N && Y[tid * RW + j] > mx) {
        mx = Y[tid * RW + j];
        arg = r;
      }
    }
    float s = 0.f;
    for (int j = 0; j < RW; ++j) {
      const int r = RW * g + j;
      if (r < a.N) s += expf(Y[tid * RW + j] - mx);
    }
    a.lm_part[(size_t)tid * a.n_groups + g] = LmPart{mx, s, arg, 0};
  }
}

template <class WT, int EPI, int RW>
__device__ __forceinline__ void run_epilogue(const GemmArgs& a, int g, int M, const float* Y) {
  if (EPI == EPI_QKV) epi_qkv<WT, RW>(a, g, M, Y);
  if (EPI == EPI_RESID) epi_resid<RW>(a, g, M, Y);
  if (EPI == EPI_SWIGLU) epi_swiglu<RW>(a, g, M, Y);
  if (EPI == EPI_LMHEAD) epi_lmhead<RW>(a, g, M, Y);
}

// Gain of 8 (bf16) or 4 (fp32) consecutive columns as floats.
template <class WT>
__device__ __forceinline__ void unpack16(const u32x4& raw, float* out) {
  if (sizeof(WT) == 2) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      out[2 * q] = __uint_as_float(raw[q] << 16);
      out[2 * q + 1] = __uint_as_float(raw[q] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) out[q] = __uint_as_float(raw[q]);
  }
}

// ----------------------------------------------------------------------------- VALU GEMV

__device__ __forceinline__ float merge_exp2(float x) { return x == -INFINITY ? 0.f : exp2f(x); }

// Split merge carried by a projection's launch (MG): polls of the merge counter before a
// projection workgroup gives up (a fraction of a second), and partial slots per lane per round.
constexpr unsigned kMgSpin = 1u << 18;
constexpr int kMgPer = 16;

// U: chunks of every row in flight per thread (one pass covers U x blockDim chunks).
// MG: the activation rows are the attention output o that the launch's first mg.nwg
// workgroups produce (k_gemv_merged): read with device-scope loads once the workgroup's
// replica of the layer's merge counter has reached the plan's target, which the first pass
// waits for after issuing its weight loads.  Those loads start about 1.7 us into the
// workgroup, so that the merge's partial loads, stores and counter updates are not queued
// behind the projection's weight stream (7B shape, 64 counter copies: the projection with the
// merge 10.3 us with this delay, 10.9-11.0 us with 0.4-0.85 us).  g: the row group.
template <class WT, int M, int EPI, int RW, int U, bool MG>
__device__ __forceinline__ void gemv_body(const GemmArgs& a, const MergeArgs& mg, const int g) {
  constexpr int RWP = RW <= 4 ? 4 : (RW <= 8 ? 8 : 16);  // RW padded to a power of two
  constexpr int CH = 16 / (int)sizeof(WT);  // elements per 16-byte load
  constexpr int NV = RW * M + M;            // per-wave totals: outputs, then sums of squares
  const int T = blockDim.x;                 // 256, or 512 for long rows
  const int nw = T >> 6;
  __shared__ float s_red[kGemvMaxThreads / 64][NV];
  __shared__ float Y[M * RW];
  __shared__ float s_scale[M];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  constexpr bool norm = EPI != EPI_RESID;  // every other epilogue follows an RMSNorm (gain checked at launch)
  const int nch = a.K / CH;
  const char* wp[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) wp[r] = weight_row<WT, EPI, RW>(a, g, r);
  const float* xr[M];
#pragma unroll
  for (int m = 0; m < M; ++m) xr[m] = a.x + (size_t)a_src_row(a, m) * a.ldx;
  float acc[RW][M], sq[M];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    sq[m] = 0.f;
#pragma unroll
    for (int r = 0; r < RW; ++r) acc[r][m] = 0.f;
  }
  constexpr bool kPre = EPI == EPI_QKV || EPI == EPI_RESID;  // at most one item per thread here
  // The epilogue's first inputs load ahead of the weight stream, the position-addressed ones
  // right behind its first loads; nothing waits for them until the epilogue.
  EpiItem item;
  if (kPre) epi_fetch_a<WT, EPI, RW>(a, g, M, tid, item);
  int mg_fail = 0;  // MG, thread 0: the merge counter never reached its target
  const __amdgpu_buffer_rsrc_t ro = dev_rsrc(MG ? a.x : nullptr, MG ? mg.o_bytes : 0u);  // o (MG only)
  // One pass over chunks c0 and c0 + T of every row.  All loads come first and none is
  // conditional (a chunk past the end re-reads the last one and leaves the sums as they
  // are), so the waits before each use count exactly; the first pass is peeled so that the
  // weight stream never waits behind the epilogue's loads at a loop header.
  auto pass = [&](int c0, auto first) {
    if constexpr (MG && decltype(first)::value) __builtin_amdgcn_s_sleep(64);  // 4096 cycles
    u32x4 wv[U][RW];
    float4 xv[U][M][CH / 4];
    u32x4 gv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = min(c0 + u * T, nch - 1);
#pragma unroll
      for (int r = 0; r < RW; ++r) wv[u][r] = ld_nt16(wp[r] + (size_t)c * 16);
      if constexpr (!MG) {
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
          for (int e4 = 0; e4 < CH / 4; ++e4) xv[u][m][e4] = *(const float4*)(xr[m] + c * CH + 4 * e4);
        if (norm) gv[u] = *(const u32x4*)((const char*)a.gain + (size_t)c * 16);
      }
    }
    if constexpr (MG) {
      if constexpr (decltype(first)::value) {
        // thread 0 polls (its poll returns after its own weight loads: loads complete in
        // order), the others wait at the barrier with their weight loads in flight
        if (tid == 0) {
          const unsigned target = a.plan->merge_target;
          unsigned it = 0;
          const unsigned* cnt = mg.cnt + (g % kMgReplicas) * kKsCntStride;
          while ((int)(__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - target) < 0) {
            if (++it == kMgSpin) {
              mg_fail = 1;
              break;
            }
            __builtin_amdgcn_s_sleep(2);
          }
        }
        __builtin_amdgcn_s_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);  // no o load moves above the wait
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = min(c0 + u * T, nch - 1);
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
          for (int e4 = 0; e4 < CH / 4; ++e4) {
            const f32x4 t = ld_dev16(ro, (uint32_t)((m * a.ldx + c * CH + 4 * e4) * 4));
            xv[u][m][e4] = make_float4(t[0], t[1], t[2], t[3]);
          }
      }
    }
    // every load above is issued before any use (the scheduler would otherwise trade loads
    // in flight for registers)
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (decltype(first)::value && kPre) epi_fetch_b<WT, EPI, RW>(a, g, item);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool valid = c0 + u * T < nch;
      float gf[CH];
      if (norm) unpack16<WT>(gv[u], gf);
#pragma unroll
      for (int m = 0; m < M; ++m) {
        float xe[CH];
#pragma unroll
        for (int e4 = 0; e4 < CH / 4; ++e4) {
          xe[4 * e4 + 0] = xv[u][m][e4].x;
          xe[4 * e4 + 1] = xv[u][m][e4].y;
          xe[4 * e4 + 2] = xv[u][m][e4].z;
          xe[4 * e4 + 3] = xv[u][m][e4].w;
        }
        if (norm) {
          float q2 = sq[m];
#pragma unroll
          for (int e = 0; e < CH; ++e) {
            q2 = fmaf(xe[e], xe[e], q2);
            xe[e] *= gf[e];
          }
          sq[m] = valid ? q2 : sq[m];
        }
#pragma unroll
        for (int r = 0; r < RW; ++r) {
          float s = acc[r][m];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (sizeof(WT) == 2) {
              s = fmaf(__uint_as_float(wv[u][r][q] << 16), xe[2 * q], s);
              s = fmaf(__uint_as_float(wv[u][r][q] & 0xffff0000u), xe[2 * q + 1], s);
            } else {
              s = fmaf(__uint_as_float(wv[u][r][q]), xe[q], s);
            }
          }
          acc[r][m] = valid ? s : acc[r][m];
        }
      }
    }
  };
  pass(tid, std::true_type{});
  for (int c0 = tid + U * T; c0 < nch; c0 += U * T) pass(c0, std::false_type{});
  // wave totals, then the waves in fixed order
#pragma unroll
  for (int m = 0; m < M; ++m) {
    float vv[RWP];
#pragma unroll
    for (int r = 0; r < RWP; ++r) vv[r] = r < RW ? acc[r][m] : 0.f;
    const float t = transpose_reduce<RWP>(vv, l);
    const int ti = transpose_index<RWP>(l);
    if ((l & (64 / RWP - 1)) == 0 && ti < RW) s_red[w][ti * M + m] = t;
    if (norm) {
      const float s = wave_sum(sq[m]);
      if (l == 0) s_red[w][RW * M + m] = s;
    }
  }
  __shared__ int s_fail;
  if (MG && tid == 0) s_fail = mg_fail;
  __syncthreads();
  if (norm && tid < M) {
    float s = 0.f;
    for (int v = 0; v < nw; ++v) s += s_red[v][RW * M + tid];
    s_scale[tid] = rsqrtf(s / (float)a.K + a.eps);
  }
  __syncthreads();
  if (tid < RW * M) {
    const int r = tid / M, m = tid - r * M;
    float v = 0.f;
    for (int q = 0; q < nw; ++q) v += s_red[q][tid];
    Y[m * RW + r] = norm ? v * s_scale[m] : v;
    if (MG && s_fail) Y[m * RW + r] = __builtin_nanf("");  // a merge that never arrived shows as NaN
  }
  __syncthreads();
  if (kPre)
    epi_apply<WT, EPI, RW>(a, g, item, Y);
  else
    run_epilogue<WT, EPI, RW>(a, g, M, Y);
}

template <class WT, int M, int EPI, int RW, int U>
__global__ __launch_bounds__(kGemvMaxThreads) void k_gemv(GemmArgs a) {
  gemv_body<WT, M, EPI, RW, U, false>(a, MergeArgs{}, blockIdx.x);
}

// The split merge of (row b / hq, query head b % hq) in a projection's launch: o = sum_s O_s
// 2^(m_s - M) / sum_s l_s 2^(m_s - M) over the row's slots, as k_attn_merge combines them (HD/4
// lanes per slot, 16-byte loads, each wave's slots across its lanes, the waves in LDS in fixed
// order), in rounds of kMgPer slots per lane (one round for up to 128 slots from 4 waves).  o
// goes out with device-scope stores; then every replica of the layer's counter is bumped (one
// per lane of wave 0), also by the workgroups of rows whose attention wrote o directly.
template <int HD>
__device__ void merge_part(const MergeArgs& mg, const Plan* plan, float* o, int b) {
  constexpr int LPS = HD / 4, SPW = 64 / LPS;
  __shared__ float s_m[kGemvMaxThreads / 64], s_l[kGemvMaxThreads / 64];
  __shared__ __align__(16) float s_o[kGemvMaxThreads / 64][HD];
  const int nw = blockDim.x >> 6, spp = SPW * nw;
  const int row = b / mg.hq, head = b - row * mg.hq;
  const int v = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int d4 = l % LPS, sl = l / LPS;
  const int kvh = head / mg.G, gi = head - kvh * mg.G;
  const size_t ncols = (size_t)mg.max_rows * mg.G;
  const size_t col = (size_t)row * mg.G + gi;
  const int nwg = plan->row_nslots[row];
  if (nwg > 1) {
    float M = -INFINITY, L = 0.f;
    f32x4 O = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < nwg; s0 += kMgPer * spp) {
      // every load of the round issued together; slots past the launch's bound re-read the
      // last one, slots past the row's count are dropped below
      float mv[kMgPer], lv[kMgPer];
      f32x4 ov[kMgPer];
#pragma unroll
      for (int i = 0; i < kMgPer; ++i) {
        const int slot = min(s0 + spp * i + SPW * v + sl, mg.nslots - 1);
        const size_t sb = ((size_t)(kvh * kAttnMaxWG + slot)) * ncols + col;
        const float2 ml = *(const float2*)(mg.ml + sb * 2);
        mv[i] = ml.x;
        lv[i] = ml.y;
        ov[i] = *(const f32x4*)(mg.part + sb * HD + 4 * d4);
      }
#pragma unroll
      for (int i = 0; i < kMgPer; ++i)
        if (s0 + spp * i + SPW * v + sl >= nwg) {
          mv[i] = -INFINITY;
          lv[i] = 0.f;
          ov[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      float Mr = M;
#pragma unroll
      for (int i = 0; i < kMgPer; ++i) Mr = fmaxf(Mr, mv[i]);
      Mr = wave_max(Mr);
      if (Mr != -INFINITY) {  // wave-uniform
        const float c = merge_exp2(M - Mr);  // earlier rounds (0 while M is -inf)
        L *= c;
        O *= c;
#pragma unroll
        for (int i = 0; i < kMgPer; ++i) {
          const float f = merge_exp2(mv[i] - Mr);
          L += lv[i] * f;
          O += ov[i] * f;
        }
        M = Mr;
      }
    }
    if constexpr (SPW == 4) {
      L = sum_x16(L);
#pragma unroll
      for (int q = 0; q < 4; ++q) O[q] = sum_x16(O[q]);
    }
    L = sum_x32(L);
#pragma unroll
    for (int q = 0; q < 4; ++q) O[q] = sum_x32(O[q]);
    if (l < LPS) *(f32x4*)&s_o[v][4 * d4] = O;
    if (l == 0) {
      s_m[v] = M;
      s_l[v] = L;
    }
    __syncthreads();
    if ((int)threadIdx.x < LPS) {  // wave 0
      float Mt = -INFINITY;
      for (int u = 0; u < nw; ++u) Mt = fmaxf(Mt, s_m[u]);
      float Lt = 0.f;
      f32x4 Ot = {0.f, 0.f, 0.f, 0.f};
      for (int u = 0; u < nw; ++u) {
        const float f = merge_exp2(s_m[u] - Mt);
        Lt += s_l[u] * f;
        Ot += *(const f32x4*)&s_o[u][4 * threadIdx.x] * f;
      }
      const __amdgpu_buffer_rsrc_t ro = dev_rsrc(o, mg.o_bytes);
      st_dev16(ro, (uint32_t)((((size_t)row * mg.hq + head) * HD + 4 * threadIdx.x) * 4), Ot / Lt);
    }
  }
  static_assert(kMgReplicas == 64, "one replica per lane of wave 0");
  if (threadIdx.x < 64) {  // wave 0: its stores complete, then the arrival
    wait_mem();
    __hip_atomic_fetch_add(mg.cnt + threadIdx.x * kKsCntStride, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// A residual projection (VALU path, M rows) whose first mg.nwg workgroups merge the attention
// splits that produce its activation rows (see MergeArgs).  The merge workgroups come first in
// the grid, so they are dispatched before any projection workgroup waits for them.
template <class WT, int M, int RW, int U>
__global__ __launch_bounds__(kGemvMaxThreads) void k_gemv_merged(GemmArgs a, MergeArgs mg) {
  if ((int)blockIdx.x < mg.nwg) {
    if (mg.hd == 128)
      merge_part<128>(mg, a.plan, const_cast<float*>(a.x), blockIdx.x);
    else
      merge_part<64>(mg, a.plan, const_cast<float*>(a.x), blockIdx.x);
    return;
  }
  gemv_body<WT, M, EPI_RESID, RW, U, true>(a, mg, (int)blockIdx.x - mg.nwg);
}

// ----------------------------------------------------------------------------- MFMA GEMM

// A workgroup computes NR consecutive 16-row groups; its W waves split K in blocks of four
// 32-column steps (so a wave reads 256 contiguous bytes of every row it streams).  Each
// activation fragment is split into bf16 hi/lo once per step and used for all NR groups,
// which is what keeps the per-step load and VALU work small when M is small.
// Row groups per workgroup allowed with MT 16-row activation tiles: four only for 2-3
// tiles (with 4 tiles their reduction slots would leave one workgroup per CU).
template <int MT>
constexpr bool mfma_nr_ok(int nr) {
  return nr == 1 || nr == 2 || (nr == 4 && MT >= 2 && MT <= 3);
}
// Waves of an MFMA workgroup at most: several row groups over several tiles keep 4 waves, so
// that the per-wave reduction slots fit in LDS.
template <int MT, int NR>
constexpr int mfma_wmax() {
  return NR >= 2 && MT >= 2 ? 4 : kMfmaMaxWaves;
}

// K shares of a residual projection (a.ksplit workgroups per block of row groups, share ks
// here): this workgroup's partial sums of its nlive groups (Y: [group][row][RW], YN apart) go to
// kpart.  Without counters (a.kcnt null) that is all: k_ksplit_reduce adds the shares to h.
// With them, the stores are device-scope ones, which other XCDs see once they have completed,
// and the workgroup then counts its arrival with a device-scope atomic; the last of the
// block's workgroups to arrive reads every share back (device-scope loads), adds them in share
// order and adds the sum to h, as the reduce kernel would, then re-arms the counter.
template <int RW>
__device__ void ksplit_finish(const GemmArgs& a, int ks, int blk, int g0, int nlive, int M, const float* Y, int YN) {
  static_assert(RW % 4 == 0, "16-byte chunks of a group's rows");
  constexpr int C4 = RW / 4;
  const int ksplit = a.ksplit;
  if (a.kcnt == nullptr) {  // k_ksplit_reduce adds the shares
    for (int r = 0; r < nlive; ++r)
      for (int i = threadIdx.x; i < M * RW; i += blockDim.x) {
        const int m = i / RW, row = RW * (g0 + r) + (i - m * RW);
        a.kpart[((size_t)ks * M + m) * a.N + row] = Y[r * YN + i];
      }
    return;
  }
  const __amdgpu_buffer_rsrc_t rk = dev_rsrc(a.kpart, (uint32_t)((size_t)ksplit * M * a.N * 4));
  for (int r = 0; r < nlive; ++r)
    for (int i = threadIdx.x; i < M * C4; i += blockDim.x) {
      const int m = i / C4, row = RW * (g0 + r) + 4 * (i - m * C4);
      const float* y = Y + r * YN + m * RW + (row - RW * (g0 + r));
      st_dev16(rk, (uint32_t)((((size_t)ks * M + m) * a.N + row) * 4), f32x4{y[0], y[1], y[2], y[3]});
    }
  wait_mem();
  __syncthreads();
  __shared__ unsigned s_tk;
  unsigned* cnt = a.kcnt + (size_t)blk * kKsCntStride;
  if (threadIdx.x == 0) s_tk = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_tk != (unsigned)(ksplit - 1)) return;
  for (int r = 0; r < nlive; ++r)
    for (int i = threadIdx.x; i < M * C4; i += blockDim.x) {
      const int m = i / C4, row = RW * (g0 + r) + 4 * (i - m * C4);
      f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int k = 0; k < ksplit; ++k) sum += ld_dev16(rk, (uint32_t)((((size_t)k * M + m) * a.N + row) * 4));
      f32x4* hp = (f32x4*)(a.h + (size_t)m * a.N + row);
      *hp = *hp + sum;
    }
  if (threadIdx.x == 0) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <class WT, int MT, int EPI, int NR>
__global__ __launch_bounds__(64 * kMfmaMaxWaves) void k_gemm_mfma(GemmArgs a) {
  constexpr int RW = rows_per_group(EPI, true);
  constexpr int NLD = (int)sizeof(WT) / 2;  // 16-byte loads per step (bf16: 1, fp32: 2)
  // steps kept in flight per wave
  constexpr int U = MT == 1 ? (NR == 1 ? 6 : 4) : (MT == 2 && NR <= 2 ? 4 : 2);
  constexpr int WMAX = mfma_wmax<MT, NR>();
  constexpr int YN = 16 * MT * RW;                   // outputs of one group
  const int W = blockDim.x >> 6;                     // waves splitting K
  __shared__ float s_red[WMAX][NR * YN];
  __shared__ float s_sq[WMAX][16 * MT];
  __shared__ float Y[NR * YN];
  __shared__ float s_scale[16 * MT];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int ksplit = EPI == EPI_RESID && a.ksplit > 1 ? a.ksplit : 1;  // K shares of a row group (adjacent workgroups)
  const int ks = (int)blockIdx.x % ksplit;
  const int g0 = (int)blockIdx.x / ksplit * NR;
  const int nlive = min(NR, a.n_groups - g0);  // groups past n_groups read clamped rows, unused
  const int M = a.M;
  const bool norm = a.gain != nullptr;
  const int n = l & 15, kg = 8 * (l >> 4);
  const char* wp[NR];  // row-major: this lane's row; tiled: this lane's bytes in the group's first block
  constexpr int BLK = 1024 * NLD;
  const bool tiled = a.wtile != nullptr;
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int g = g0 + (r < nlive ? r : 0);
    wp[r] = tiled ? a.wtile + (size_t)g * a.tsteps * BLK + 16 * l : weight_row<WT, EPI, RW>(a, g, n);
  }
  const float* xr[MT];
  bool own[MT];  // this lane's A row is a real row (rows past M repeat row M-1)
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    own[mt] = 16 * mt + n < M;
    xr[mt] = a.x + (size_t)a_src_row(a, min(16 * mt + n, M - 1)) * a.ldx;
  }
  // This workgroup's 32-column steps [s0, s1): all of K, or a share of whole 4-step blocks.
  const int nsteps_all = (a.K + 31) >> 5;
  const int sps = ksplit > 1 ? (((nsteps_all + ksplit - 1) / ksplit + 3) & ~3) : nsteps_all;
  const int s0 = ks * sps, s1 = min(nsteps_all, s0 + sps);
  const int kend = min(a.K, 32 * s1);
  const int nblk = (max(s1 - s0, 0) + 3) >> 2;
  const int niter = nblk > w ? 4 * ((nblk - w + W - 1) / W) : 0;  // this wave's steps
  auto step_of = [&](int it) { return s0 + 4 * (w + W * (it >> 2)) + (it & 3); };
  f32x4 acc[NR][MT];
  float sq[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    sq[mt] = 0.f;
#pragma unroll
    for (int r = 0; r < NR; ++r) acc[r][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // K offset of this lane's 8 elements at iteration it, or -1 past the end of K
  auto kof = [&](int it) {
    const int k = 32 * step_of(it) + kg;
    return k < kend ? k : -1;
  };
  // Every operand of a step (weights, activations, gain) is loaded U steps ahead of its use.
  struct Step {
    u32x4 wv[NR][NLD];
    u32x4 gv[NLD];
    float4 xv[MT][2];
  };
  auto issue = [&](int it, Step& st) {
    const int k = kof(it), kk = k < 0 ? 0 : k;
    const size_t woff = tiled ? (size_t)(k < 0 ? 0 : step_of(it)) * BLK : (size_t)kk * sizeof(WT);
    const int qs = tiled ? 1024 : 16;  // offset of a lane's second 16 bytes (fp32)
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
      for (int q = 0; q < NLD; ++q) st.wv[r][q] = ld_nt16(wp[r] + woff + qs * q);
    if (norm)
#pragma unroll
      for (int q = 0; q < NLD; ++q) st.gv[q] = *(const u32x4*)((const char*)a.gain + (size_t)kk * sizeof(WT) + 16 * q);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      st.xv[mt][0] = *(const float4*)(xr[mt] + kk);
      st.xv[mt][1] = *(const float4*)(xr[mt] + kk + 4);
    }
  };
  // The MFMAs of one step from its operands (k < 0: past the end of K, contributes zero;
  // checked only when `checkc` is true, i.e. in the tail steps).
  auto compute = [&](const Step& cur, int k, auto checkc) {
    constexpr bool check = decltype(checkc)::value;
    bf16x8 bhi[NR], blo[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      if (NLD == 1) {
        bhi[r] = __builtin_bit_cast(bf16x8, cur.wv[r][0]);
      } else {
        u32x4 ph, pl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint16_t h0, l0, h1, l1;
          split_bf16(__uint_as_float(cur.wv[r][q >> 1][(q & 1) * 2 + 0]), h0, l0);
          split_bf16(__uint_as_float(cur.wv[r][q >> 1][(q & 1) * 2 + 1]), h1, l1);
          ph[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
          pl[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        }
        bhi[r] = __builtin_bit_cast(bf16x8, ph);
        blo[r] = __builtin_bit_cast(bf16x8, pl);
      }
    }
    float gf[8];
    if (norm) {
      unpack16<WT>(cur.gv[0], gf);
      if (sizeof(WT) == 4) unpack16<WT>(cur.gv[NLD - 1], gf + 4);
    }
    const bool live = !check || k >= 0;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const float4 x0 = cur.xv[mt][0], x1 = cur.xv[mt][1];
      float xe[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
      if (check)
#pragma unroll
        for (int e = 0; e < 8; ++e) xe[e] = live ? xe[e] : 0.f;
      if (norm) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sq[mt] = fmaf(xe[e], xe[e], sq[mt]);
          xe[e] *= gf[e];
        }
      }
      u32x4 ph, pl;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t h, lo;
        split_trunc2(xe[2 * q], xe[2 * q + 1], h, lo);
        ph[q] = h;
        pl[q] = lo;
      }
      const bf16x8 ahi = __builtin_bit_cast(bf16x8, ph), alo = __builtin_bit_cast(bf16x8, pl);
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        acc[r][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bhi[r], acc[r][mt], 0, 0, 0);
        acc[r][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bhi[r], acc[r][mt], 0, 0, 0);
        if (NLD == 2) acc[r][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, blo[r], acc[r][mt], 0, 0, 0);
      }
    }
  };
  Step buf[U];
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (u < niter) issue(u, buf[u]);
  // Steps whose 32 columns all lie inside K need no end check; they come first.  With K a
  // multiple of 128 (all model shapes but the tiny one) that is every step.
  int nfull = niter;
  while (nfull > 0 && step_of(nfull - 1) >= min(a.K >> 5, s1)) --nfull;
  using Check = std::integral_constant<bool, true>;
  using NoCheck = std::integral_constant<bool, false>;
  int it0 = 0;
  // steady state: U whole steps per trip, each buffer refilled right after its use
  for (; it0 + U <= nfull; it0 += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      compute(buf[u], kof(it0 + u), NoCheck{});
      if (it0 + u + U < niter) issue(it0 + u + U, buf[u]);
    }
  }
  // remaining steps (fewer than U whole steps, then partial ones): operands already issued
  for (; it0 < niter; it0 += U) {
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (it0 + u < niter) {
        compute(buf[u], kof(it0 + u), Check{});
        if (it0 + u + U < niter) issue(it0 + u + U, buf[u]);
      }
  }
  // lane (n, l/16): acc[r][mt][i] = Y_r[m = 16mt + 4(l/16) + i][n]; sq over the lanes of row n
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
      for (int i = 0; i < 4; ++i) s_red[w][r * YN + (16 * mt + 4 * (l >> 4) + i) * RW + n] = acc[r][mt][i];
    if (norm) {
      float s = own[mt] ? sq[mt] : 0.f;
      s = sum_x16(s);
      s = sum_x32(s);
      if (l < 16) s_sq[w][16 * mt + n] = s;
    }
  }
  __syncthreads();
  if (norm && tid < M) {
    float s = 0.f;
    for (int v = 0; v < W; ++v) s += s_sq[v][tid];
    s_scale[tid] = rsqrtf(s / (float)a.K + a.eps);
  }
  __syncthreads();
  for (int idx = tid; idx < NR * YN; idx += blockDim.x) {
    const int j = idx % YN;
    if (j >= M * RW) continue;
    float v = 0.f;
    for (int q = 0; q < W; ++q) v += s_red[q][idx];
    Y[idx] = norm ? v * s_scale[j / RW] : v;
  }
  __syncthreads();
  if (EPI == EPI_RESID && ksplit > 1) {  // partial sums of this K share (no norm on this path)
    ksplit_finish<RW>(a, ks, (int)blockIdx.x / ksplit, g0, nlive, M, Y, YN);
    return;
  }
  for (int r = 0; r < nlive; ++r) run_epilogue<WT, EPI, RW>(a, g0 + r, M, Y + r * YN);
}

// ----------------------------------------------------------------------------- MFMA GEMM, row waves

// The K-split kernel above reads every activation row once per workgroup, besides its one or
// two row groups' weights; with several 16-row activation tiles that is most of what a
// workgroup reads.  Here the 4 waves of a workgroup own different row groups (NRW each, 4 NRW
// in all) over the whole of the workgroup's K range, and the activations are staged once per
// workgroup in LDS, in 128-column chunks: loaded from global, scaled by the norm gain, split
// into bf16 hi/lo and written in MFMA fragment order, while the previous chunk is multiplied.
// So a workgroup reads its activations once for 4 NRW row groups.  Each wave sums its K range
// in step order (one MFMA chain per group and tile); K shares (residual projections) go
// through the K-share partials as in the kernel above.
constexpr int kRwSteps = 4;  // 32-column steps per staged activation chunk
#ifndef LASER_RW_RING
#define LASER_RW_RING 8
#endif
constexpr int kRwRing = LASER_RW_RING;  // bf16 weight steps in flight per wave (fp32: half)

template <class WT, int MT, int EPI, int NRW>
__global__ __launch_bounds__(256) void k_gemm_mfma_rw(GemmArgs a) {
  constexpr int RW = rows_per_group(EPI, true);
  constexpr int NLD = (int)sizeof(WT) / 2;  // 16-byte weight loads per step (bf16: 1, fp32: 2)
  constexpr int CS = kRwSteps, U = kRwRing / NLD < 2 * CS ? 2 * CS : kRwRing / NLD;
  constexpr int NQ = U / CS;  // chunks per turn of the weight ring
  static_assert(U % CS == 0 && NQ % 2 == 0, "whole chunks per ring turn, two activation buffers");
  static_assert(CS == 4, "each of the 4 waves stages one step of a chunk");
  constexpr int NG = 4 * NRW;                 // row groups of the workgroup
  constexpr int YN = 16 * MT * RW;            // outputs of one group
  constexpr int ABUF = MT * CS * 2 * 1024;    // one staged chunk: tiles x steps x (hi, lo) x 1 KB
  constexpr int YBYTES = NG * YN * 4;
  constexpr int SMEM = 2 * ABUF > YBYTES ? 2 * ABUF : YBYTES;
  __shared__ __align__(16) char smem[SMEM];  // two activation chunks; after the loop, Y
  __shared__ float s_sqp[4][16 * MT], s_scale[16 * MT];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int ksplit = EPI == EPI_RESID && a.ksplit > 1 ? a.ksplit : 1;
  const int ks = (int)blockIdx.x % ksplit;
  const int gw0 = (int)blockIdx.x / ksplit * NG;  // the workgroup's first group
  const int M = a.M;
  constexpr bool norm = EPI != EPI_RESID;  // every other epilogue follows an RMSNorm (gain checked at launch)
  const int n = l & 15;
  const bool tiled = a.wtile != nullptr;
  constexpr int BLK = 1024 * NLD;
  const char* wp[NRW];  // this lane's bytes of its wave's groups (groups past n_groups: clamped, not stored)
#pragma unroll
  for (int r = 0; r < NRW; ++r) {
    const int g = min(gw0 + w * NRW + r, a.n_groups - 1);
    wp[r] = tiled ? a.wtile + (size_t)g * a.tsteps * BLK + 16 * l : weight_row<WT, EPI, RW>(a, g, n);
  }
  // the workgroup's 32-column steps [s0, s1): all of K, or a share of whole chunks
  const int nsteps_all = (a.K + 31) >> 5;
  const int sps = ksplit > 1 ? ((nsteps_all + ksplit - 1) / ksplit + CS - 1) / CS * CS : nsteps_all;
  const int s0 = ks * sps, s1 = min(nsteps_all, s0 + sps);
  const int nst = max(s1 - s0, 0);
  const int nch = (nst + CS - 1) / CS;
  const int kend = min(a.K, 32 * s1);

  // Staging: wave w stages step w of the chunk, lane l the operand of fragment lane l: row
  // 16 mt + l % 16 of every tile, columns 32 w + 8 (l / 16) .. + 7.  So each wave's LDS
  // writes are 1 KB contiguous (no bank conflicts).
  const int srow = l & 15, sc8 = 32 * w + 8 * (l >> 4);
  const int sj = w, slane = l;
  const float* xs[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) xs[mt] = a.x + (size_t)a_src_row(a, min(16 * mt + srow, M - 1)) * a.ldx;
  float4 xv[MT][2];
  u32x4 gv[NLD];
  float sq[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) sq[mt] = 0.f;
  // column of this thread's 8 values in chunk c (-1: past the end of K); chunks past the
  // last reload the last one (in bounds, unused)
  auto scol = [&](int c) {
    const int k = 32 * (s0 + min(c, nch - 1) * CS) + sc8;
    return k < kend ? k : -1;
  };
  auto aload = [&](int c) {
    const int k = scol(c), kk = k < 0 ? 0 : k;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      xv[mt][0] = *(const float4*)(xs[mt] + kk);
      xv[mt][1] = *(const float4*)(xs[mt] + kk + 4);
    }
    if (norm)
#pragma unroll
      for (int q = 0; q < NLD; ++q) gv[q] = *(const u32x4*)((const char*)a.gain + (size_t)kk * sizeof(WT) + 16 * q);
  };
  auto astore = [&](int c, auto bufc) {
    constexpr int buf = decltype(bufc)::value;
    const bool live = scol(c) >= 0;
    float gf[8];
    if (norm) {
      unpack16<WT>(gv[0], gf);
      if (sizeof(WT) == 4) unpack16<WT>(gv[NLD - 1], gf + 4);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const float4 x0 = xv[mt][0], x1 = xv[mt][1];
      float xe[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) xe[e] = live ? xe[e] : 0.f;
      if (norm) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          sq[mt] = fmaf(xe[e], xe[e], sq[mt]);
          xe[e] *= gf[e];
        }
      }
      u32x4 ph, pl;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t h, lo;
        split_trunc2(xe[2 * q], xe[2 * q + 1], h, lo);
        ph[q] = h;
        pl[q] = lo;
      }
      char* dst = smem + buf * ABUF + ((mt * CS + sj) * 2) * 1024 + 16 * slane;
      *(u32x4*)dst = ph;
      *(u32x4*)(dst + 1024) = pl;
    }
  };

  // weights: a ring of U steps; steps past the last reload the last one (in bounds, unused)
  u32x4 wv[U][NRW][NLD];
  auto wissue = [&](int it, auto slotc) {
    constexpr int slot = decltype(slotc)::value;
    const int st = s0 + min(it, nst - 1);
    const int k = 32 * st + 8 * (l >> 4);
    const size_t woff = tiled ? (size_t)st * BLK : (size_t)(k < kend ? k : 0) * sizeof(WT);
    const int qs = tiled ? 1024 : 16;
#pragma unroll
    for (int r = 0; r < NRW; ++r)
#pragma unroll
      for (int q = 0; q < NLD; ++q) wv[slot][r][q] = ld_nt16(wp[r] + woff + qs * q);
  };
  f32x4 acc[NRW][MT];
#pragma unroll
  for (int r = 0; r < NRW; ++r)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[r][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](auto slotc, auto bufc, auto jc) {
    constexpr int slot = decltype(slotc)::value, buf = decltype(bufc)::value, j = decltype(jc)::value;
    bf16x8 bhi[NRW], blo[NRW];
#pragma unroll
    for (int r = 0; r < NRW; ++r) {
      if (NLD == 1) {
        bhi[r] = __builtin_bit_cast(bf16x8, wv[slot][r][0]);
      } else {
        u32x4 ph, pl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint16_t h0, l0, h1, l1;
          split_bf16(__uint_as_float(wv[slot][r][q >> 1][(q & 1) * 2 + 0]), h0, l0);
          split_bf16(__uint_as_float(wv[slot][r][q >> 1][(q & 1) * 2 + 1]), h1, l1);
          ph[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
          pl[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        }
        bhi[r] = __builtin_bit_cast(bf16x8, ph);
        blo[r] = __builtin_bit_cast(bf16x8, pl);
      }
    }
    bf16x8 ahi[MT], alo[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const char* src = smem + buf * ABUF + ((mt * CS + j) * 2) * 1024 + 16 * l;
      ahi[mt] = *(const bf16x8*)src;
      alo[mt] = *(const bf16x8*)(src + 1024);
    }
    // every accumulator's hi product, then every lo product: consecutive matrix-core ops
    // feed different accumulators (each accumulator still sums hi before lo)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < NRW; ++r)
        acc[r][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[mt], bhi[r], acc[r][mt], 0, 0, 0);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < NRW; ++r)
        acc[r][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[mt], bhi[r], acc[r][mt], 0, 0, 0);
    if (NLD == 2)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < NRW; ++r)
          acc[r][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi[mt], blo[r], acc[r][mt], 0, 0, 0);
  };
  // chunk c (the q-th of a ring turn): its CS steps from LDS buffer q % 2 (ring slots q*CS ..),
  // each slot refilled U steps ahead; then the next chunk's activations (loaded a chunk ago)
  // go to the other buffer, and the one after is loaded.  `checked`: the last chunks, where
  // steps and chunks may be missing; elsewhere nothing is conditional, so that no load waits
  // for a later one at a branch merge (vector-memory counters complete in order).
  auto chunk = [&](int c, auto qc, auto checkedc) {
    constexpr int q = decltype(qc)::value, buf = q & 1;
    constexpr bool checked = decltype(checkedc)::value;
    static_for<CS>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
      const int it = c * CS + j;
      if (!checked || it < nst) {
        compute(std::integral_constant<int, q * CS + j>{}, std::integral_constant<int, buf>{}, jc);
        wissue(it + U, std::integral_constant<int, q * CS + j>{});
      }
    });
    if (!checked || c + 1 < nch) astore(c + 1, std::integral_constant<int, buf ^ 1>{});
    __syncthreads();
    if (!checked || c + 2 < nch) aload(c + 2);
  };
  if (nch > 0) {
    aload(0);
    astore(0, std::integral_constant<int, 0>{});
    if (nch > 1) aload(1);
    static_for<U>([&](auto u) { wissue((int)decltype(u)::value, u); });
    __syncthreads();
    int c = 0;
    // whole ring turns whose chunks are full and followed by two more chunks
    for (; c + NQ + 1 < nch; c += NQ)
      static_for<NQ>([&](auto q) { chunk(c + (int)decltype(q)::value, q, std::false_type{}); });
    for (; c < nch; c += NQ)
      static_for<NQ>([&](auto q) {
        if (c + (int)decltype(q)::value < nch) chunk(c + (int)decltype(q)::value, q, std::true_type{});
      });
  }
  // the rows' sums of squares: lanes l, l ^ 16, l ^ 32, l ^ 48 of every wave hold row l % 16
  if (norm) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float v = sq[mt];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (l < 16) s_sqp[w][16 * mt + l] = v;
    }
  }
  // lane (n, l/16): acc[r][mt][i] = Y_r[m = 16mt + 4(l/16) + i][n]  (the loop ended with a barrier)
  float* Y = (float*)smem;
#pragma unroll
  for (int r = 0; r < NRW; ++r)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) Y[(w * NRW + r) * YN + (16 * mt + 4 * (l >> 4) + i) * RW + n] = acc[r][mt][i];
  __syncthreads();
  if (norm && tid < M) s_scale[tid] = rsqrtf((s_sqp[0][tid] + s_sqp[1][tid] + s_sqp[2][tid] + s_sqp[3][tid]) / (float)a.K + a.eps);
  __syncthreads();
  const int nlive = min(NG, a.n_groups - gw0);
  if (norm)
    for (int idx = tid; idx < NG * YN; idx += blockDim.x) {
      const int j = idx % YN;
      if (j < M * RW) Y[idx] *= s_scale[j / RW];
    }
  __syncthreads();
  if (EPI == EPI_RESID && ksplit > 1) {  // partial sums of this K share (no norm on this path)
    ksplit_finish<RW>(a, ks, (int)blockIdx.x / ksplit, gw0, nlive, M, Y, YN);
    return;
  }
  for (int r = 0; r < nlive; ++r) run_epilogue<WT, EPI, RW>(a, gw0 + r, M, Y + r * YN);
}

// h[i] += kpart[0][i] + kpart[1][i] + ... (K shares in order), i < M * N.
__global__ void k_ksplit_reduce(float* h, const float* kpart, int ksplit, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int k = 0; k < ksplit; ++k) s += kpart[(size_t)k * n + i];
  h[i] += s;
}

hipError_t launch_ksplit_reduce(const GemmArgs& a, hipStream_t s) {
  const int n = a.M * a.N;
  return launch_k(k_ksplit_reduce, dim3((n + 255) / 256), dim3(256), s, a.h, (const float*)a.kpart, a.ksplit, n);
}

// ----------------------------------------------------------------------------- QKV over K slices

// QKV of wide forwards (3-4 activation tiles: batched decode with riding probe rows).  In the
// K-split kernel every workgroup reads the fp32 activation rows over its K range for its one or
// two row groups: at 52 rows of the 8B shape that is three times the weight bytes.  Here a
// workgroup takes one slice of K (SS 32-column steps), stages the slice of every activation row
// once in LDS (times the norm gain, split into bf16 hi/lo in A-operand order), and its NW waves
// run gb = NW GPW row groups over it (wave w: groups w, w + NW, ...).  Every wave issues its
// share of the activation loads, then all of its groups' weight loads, before it waits for
// anything.  (Measured at 56 rows of the 8B shape: the activations that miss in L2 still arrive
// behind much of the chip's weight traffic, 5-10 us after the start, but waiting for them
// before requesting the weights is slower: 22.5 against 19.5 us.)  Each A fragment is read from
// LDS once per wave for all of its groups.  Each slice's partial sums and each row's sum of
// squares over the slice go to qpart / sqpart; k_qkv_slices_epi adds the slices in order,
// applies the norm scale, then bias, rotation and the stores of the QKV epilogue.  Weights: the tile-order copy when there is one, else the
// row-major tensors (the same products in the same order).  Partial sums: qpart[slice][m][16 g +
// n], the group order of the QKV tiles (group g holds rotary pairs 8g .. 8g+7, low dims in rows
// 0-7, high dims in rows 8-15).
template <int MT, int SS, int GPW, int NW>
__global__ __launch_bounds__(64 * NW) void k_qkv_slices(GemmArgs a, float* qpart, float* sqpart, int gb) {
  constexpr int NU = MT * SS;              // (tile, step) units of the staged slice
  constexpr int UPW = (NU + NW - 1) / NW;  // units per wave
  __shared__ __align__(16) u32x4 s_a[MT][SS][2][64];  // [tile][step][hi, lo][lane]
  __shared__ float s_sq[NU][16];                       // per unit: the 16 rows' sums of squares over its 32 columns
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int slice = blockIdx.x, g0 = blockIdx.y * gb;
  const int gend = min(g0 + gb, a.n_groups);
  const int M = a.M, K = a.K, N = a.N;
  const int k0 = slice * SS * 32;
  const int nst = a.tsteps;  // 32-column steps of the tile-order weights
  // Activation loads first, all in flight together: unit u = w + NW i is tile u / SS, step
  // u % SS; lane l holds row 16 t + l % 16, 8 columns at 32 st + 8 (l / 16).  Units past NU
  // read unit NU - 1 again (not used).  Loads through global pointers, so that the compiler
  // need not keep them behind the LDS stores.
  u32x4 xa[UPW], xb[UPW], gv[UPW];
#pragma unroll
  for (int i = 0; i < UPW; ++i) {
    const int u = min(w + NW * i, NU - 1), t = u / SS, st = u - t * SS;
    const int row = 16 * t + (l & 15), k = k0 + 32 * st + 8 * (l >> 4);
    const bool in = row < M && k < K;  // K is a multiple of 8
    const size_t off = in ? (size_t)row * a.ldx + k : 0;
    xa[i] = ld_global<u32x4>(a.x + off);
    xb[i] = ld_global<u32x4>(a.x + off + 4);
    gv[i] = ld_global<u32x4>((const char*)a.gain + (in ? (size_t)k * 2 : 0));
  }
  // Then group j of this wave (g0 + w + j NW) over the slice, from the tile-order copy (steps
  // past K read the last step) or the row-major tensors (lane l % 16's row; columns past K read
  // column 0): the A operand there is zero.  Past the workgroup's groups the last one is read
  // again (not used).
  u32x4 wv[GPW][SS];
#pragma unroll
  for (int j = 0; j < GPW; ++j) {
    const int g = min(g0 + w + j * NW, gend - 1);
    if (a.wtile) {
#pragma unroll
      for (int st = 0; st < SS; ++st)
        wv[j][st] = ld_nt16(a.wtile + ((size_t)g * nst + min(slice * SS + st, nst - 1)) * 1024 + 16 * l);
    } else {
      const char* rp = weight_row<bf16_t, EPI_QKV, 16>(a, g, l & 15);
#pragma unroll
      for (int st = 0; st < SS; ++st) {
        const int k = k0 + 32 * st + 8 * (l >> 4);
        wv[j][st] = ld_nt16(rp + (size_t)(k < K ? k : 0) * 2);
      }
    }
  }
  // staged units: A = x times the gain, split into bf16 hi / lo; rows past M and columns past K zero
#pragma unroll
  for (int i = 0; i < UPW; ++i) {
    const int u = w + NW * i;
    if (u >= NU) break;
    const int t = u / SS, st = u - t * SS;
    const int row = 16 * t + (l & 15), k = k0 + 32 * st + 8 * (l >> 4);
    const bool in = row < M && k < K;
    float gf[8];
    unpack16<bf16_t>(gv[i], gf);
    float xe[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      xe[e] = __uint_as_float(xa[i][e]);
      xe[4 + e] = __uint_as_float(xb[i][e]);
    }
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xe[e] = in ? xe[e] : 0.f;
      sq = fmaf(xe[e], xe[e], sq);
      xe[e] *= gf[e];
    }
    u32x4 ph, pl;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t h, lo;
      split_trunc2(xe[2 * q], xe[2 * q + 1], h, lo);
      ph[q] = h;
      pl[q] = lo;
    }
    s_a[t][st][0][l] = ph;
    s_a[t][st][1][l] = pl;
    sq = sum_x16(sq);  // lanes l, l+16, l+32, l+48 hold the same row
    sq = sum_x32(sq);
    if (l < 16) s_sq[u][l] = sq;
  }
  __syncthreads();
  if (tid < M) {  // the row's sum of squares over the slice, its steps in order
    const int t = tid >> 4;
    float sq = 0.f;
#pragma unroll
    for (int st = 0; st < SS; ++st) sq += s_sq[t * SS + st][tid & 15];
    sqpart[(size_t)slice * M + tid] = sq;
  }
  // each A fragment read from LDS once per wave, for all of the wave's groups;
  // acc[j][mt][i] = Y[m = 16 mt + 4 (l / 16) + i][16 g_j + l % 16]
  f32x4 acc[GPW][MT];
#pragma unroll
  for (int j = 0; j < GPW; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < SS; ++st)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const bf16x8 ahi = __builtin_bit_cast(bf16x8, s_a[mt][st][0][l]);
      const bf16x8 alo = __builtin_bit_cast(bf16x8, s_a[mt][st][1][l]);
#pragma unroll
      for (int j = 0; j < GPW; ++j) {
        const bf16x8 b = __builtin_bit_cast(bf16x8, wv[j][st]);
        acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, b, acc[j][mt], 0, 0, 0);
        acc[j][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, b, acc[j][mt], 0, 0, 0);
      }
    }
#pragma unroll
  for (int j = 0; j < GPW; ++j) {
    const int g = g0 + w + j * NW;
    if (g >= gend) break;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = 16 * mt + 4 * (l >> 4) + i;
        if (m < M) qpart[((size_t)slice * M + m) * N + 16 * g + (l & 15)] = acc[j][mt][i];
      }
  }
}

// One thread per (row, 4 consecutive rotary pairs of a group): the slices summed in order, the
// norm scale, then the QKV epilogue of each pair (bias, rotation of q and k, q stored, K/V
// appended to the row's page).
template <class WT>
__global__ __launch_bounds__(256) void k_qkv_slices_epi(GemmArgs a, const float* qpart, const float* sqpart,
                                                         int nslices) {
  const int nq = a.N / 8;  // quads of pairs per row (two per group)
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.M * nq) return;
  const int m = idx / nq, qd = idx - m * nq;
  const int g = qd >> 1, j0 = 4 * (qd & 1);
  // the row's descriptor, then what it addresses (rotations of the 4 pairs, the KV page) in
  // flight with the partial sums
  const RowDesc rd = a.plan->rows[m];
  const int i0 = qkv_pair(a, 8 * g + j0).i;  // the 4 pairs are consecutive pairs of one head
  float2 cs[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) cs[e] = a.rope[(size_t)rd.pos * (a.hd >> 1) + i0 + e];
  const int page = a.bt[(size_t)rd.seq * a.max_pps + (rd.pos >> 4)];
  float4 slo = {0.f, 0.f, 0.f, 0.f}, shi = {0.f, 0.f, 0.f, 0.f};
  float sq = 0.f;
#pragma unroll 8
  for (int s2 = 0; s2 < nslices; ++s2) {
    const float* pr = qpart + ((size_t)s2 * a.M + m) * a.N + 16 * g + j0;
    const float4 lo = *(const float4*)pr, hi = *(const float4*)(pr + 8);
    slo.x += lo.x;
    slo.y += lo.y;
    slo.z += lo.z;
    slo.w += lo.w;
    shi.x += hi.x;
    shi.y += hi.y;
    shi.z += hi.z;
    shi.w += hi.w;
    sq += sqpart[(size_t)s2 * a.M + m];
  }
  const float scale = rsqrtf(sq / (float)a.K + a.eps);
  const float vlo[4] = {slo.x, slo.y, slo.z, slo.w}, vhi[4] = {shi.x, shi.y, shi.z, shi.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const QkvPair q = qkv_pair(a, 8 * g + j0 + e);
    const int dlo = q.i, dhi = (a.hd >> 1) + q.i;
    float ylo = vlo[e] * scale, yhi = vhi[e] * scale;
    if (a.b0 != nullptr) {  // the three biases are set together
      const size_t e0 = (size_t)q.hh * a.hd + q.i, e1 = e0 + (a.hd >> 1);
      ylo += bf2f(ld_global<uint16_t>((const char*)q.bias + 2 * e0));
      yhi += bf2f(ld_global<uint16_t>((const char*)q.bias + 2 * e1));
    }
    if (q.isq || q.isk) {
      const float rlo = ylo * cs[e].x - yhi * cs[e].y;
      const float rhi = yhi * cs[e].x + ylo * cs[e].y;
      ylo = rlo;
      yhi = rhi;
    }
    if (q.isq) {
      float* qo = a.q_out + ((size_t)m * a.hq + q.hh) * a.hd;
      qo[dlo] = ylo;
      qo[dhi] = yhi;
    } else {
      const int t = rd.pos & 15;
      const size_t blk = (((size_t)a.layer * a.num_pages + page) * a.hkv + q.hh) * (size_t)(16 * a.hd);
      void* pool = q.isk ? a.kpool : a.vpool;
      const size_t olo = blk + (q.isk ? k_block_off(t, dlo) : v_block_off(t, dlo));
      const size_t ohi = blk + (q.isk ? k_block_off(t, dhi) : v_block_off(t, dhi));
      if (a.kv_fp8) {
        stw<fp8_t>(pool, olo, ylo);
        stw<fp8_t>(pool, ohi, yhi);
      } else {
        stw<WT>(pool, olo, ylo);
        stw<WT>(pool, ohi, yhi);
      }
    }
  }
}

hipError_t launch_qkv_slices(const GemmArgs& a, float* qpart, float* sqpart, hipStream_t s) {
  constexpr int SS = kQSliceSteps, GPW = 2, NW = kQSliceGroups / GPW;
  const int mt = (a.M + 15) / 16;
  if (a.gain == nullptr || a.row_map || a.N % 16 != 0 || a.n_groups * 16 != a.N || a.K % 8 != 0 ||
      a.tsteps != (a.K + 31) / 32 || mt < 3 || mt > 4)
    return hipErrorInvalidValue;
  const int nslices = (a.K + SS * 32 - 1) / (SS * 32);
  const dim3 grid(nslices, (a.n_groups + kQSliceGroups - 1) / kQSliceGroups), block(64 * NW);
  const hipError_t e =
      mt == 3 ? launch_k(k_qkv_slices<3, SS, GPW, NW>, grid, block, s, a, qpart, sqpart, (int)kQSliceGroups)
              : launch_k(k_qkv_slices<4, SS, GPW, NW>, grid, block, s, a, qpart, sqpart, (int)kQSliceGroups);
  if (e != hipSuccess) return e;
  const int n = a.M * (a.N / 8);
  return launch_k(k_qkv_slices_epi<bf16_t>, dim3((n + 255) / 256), dim3(256), s, a, (const float*)qpart,
                  (const float*)sqpart, nslices);
}

// ----------------------------------------------------------------------------- weight tiles

// One block (group g, step s) per workgroup of 64 lanes: lane (n = l % 16, q = l / 16) gets
// the 8 columns 32 s + 8 q .. + 7 of the group's row n (zeros past K), as the MFMA path's
// B operand takes them.  fp32 weights: 16 bytes at l * 16 and 16 more at 1024 + l * 16.
template <class WT, int EPI>
__global__ __launch_bounds__(64) void k_tile_weights(GemmArgs a, char* dst) {
  constexpr int NLD = (int)sizeof(WT) / 2;
  constexpr int CH = 8;  // columns per lane
  const int g = blockIdx.y, s = blockIdx.x, l = threadIdx.x;
  const int n = l & 15, k0 = 32 * s + CH * (l >> 4);
  const char* row = weight_row<WT, EPI, 16>(a, g, n);
  char* out = dst + ((size_t)g * gridDim.x + s) * (1024 * NLD) + 16 * l;
#pragma unroll
  for (int q = 0; q < NLD; ++q) {
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    const int kq = k0 + q * (CH / NLD);  // first column of these 16 bytes
    if (kq + CH / NLD <= a.K) v = *(const u32x4*)(row + (size_t)kq * sizeof(WT));
    *(u32x4*)(out + 1024 * q) = v;
  }
}

template <class WT>
static hipError_t launch_tiles(int epi, const GemmArgs& a, char* dst, hipStream_t s) {
  const dim3 grid((a.K + 31) / 32, a.n_groups);
  switch (epi) {
    case EPI_QKV: return launch_k(k_tile_weights<WT, EPI_QKV>, grid, dim3(64), s, a, dst);
    case EPI_RESID: return launch_k(k_tile_weights<WT, EPI_RESID>, grid, dim3(64), s, a, dst);
    case EPI_SWIGLU: return launch_k(k_tile_weights<WT, EPI_SWIGLU>, grid, dim3(64), s, a, dst);
    case EPI_LMHEAD: return launch_k(k_tile_weights<WT, EPI_LMHEAD>, grid, dim3(64), s, a, dst);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_tile_weights(int dtype, int epi, const GemmArgs& a, char* dst, hipStream_t s) {
  return dtype == 1 ? launch_tiles<bf16_t>(epi, a, dst, s) : launch_tiles<float>(epi, a, dst, s);
}

// ----------------------------------------------------------------------------- launch

template <class WT, int MT, int NR>
static hipError_t launch_mfma(int epi, dim3 grid, dim3 block, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_k(k_gemm_mfma<WT, MT, EPI_QKV, NR>, grid, block, s, a);
    case EPI_RESID: return launch_k(k_gemm_mfma<WT, MT, EPI_RESID, NR>, grid, block, s, a);
    case EPI_SWIGLU: return launch_k(k_gemm_mfma<WT, MT, EPI_SWIGLU, NR>, grid, block, s, a);
    case EPI_LMHEAD: return launch_k(k_gemm_mfma<WT, MT, EPI_LMHEAD, NR>, grid, block, s, a);
    default: return hipErrorInvalidValue;
  }
}

template <class WT, int MT, int NRW>
static hipError_t launch_mfma_rw(int epi, dim3 grid, const GemmArgs& a, hipStream_t s) {
  const dim3 block(256);
  switch (epi) {
    case EPI_QKV: return launch_k(k_gemm_mfma_rw<WT, MT, EPI_QKV, NRW>, grid, block, s, a);
    case EPI_RESID: return launch_k(k_gemm_mfma_rw<WT, MT, EPI_RESID, NRW>, grid, block, s, a);
    case EPI_SWIGLU: return launch_k(k_gemm_mfma_rw<WT, MT, EPI_SWIGLU, NRW>, grid, block, s, a);
    case EPI_LMHEAD: return launch_k(k_gemm_mfma_rw<WT, MT, EPI_LMHEAD, NRW>, grid, block, s, a);
    default: return hipErrorInvalidValue;
  }
}

// VALU GEMV variants built, by chunks in flight per thread: two for every row count and
// weight type; one (short rows) and three (long residual rows, at most one workgroup per
// compute unit) for bf16 weights and one or two rows, where the runtime picks them.  Four-row
// QKV groups exist only with one chunk per thread (short rows).
template <class WT, int MODE, int EPI, int RW, int U>
constexpr bool gemv_built() {
  const bool valu_bf16 = std::is_same<WT, bf16_t>::value && MODE <= 2;
  if (RW == 4) return valu_bf16 && U == 1;
  if (U == 2) return true;
  return valu_bf16 && (U == 1 || (U == 3 && EPI == EPI_RESID));
}

template <class WT, int MODE, int EPI, int RW>
static hipError_t launch_gemv_u(int u, dim3 grid, dim3 block, const GemmArgs& a, hipStream_t s) {
  switch (u) {
#define LASER_GEMV_U(UU)                                                               \
  case UU:                                                                             \
    if constexpr (gemv_built<WT, MODE, EPI, RW, UU>())                                 \
      return launch_k(k_gemv<WT, MODE, EPI, RW, UU>, grid, block, s, a);               \
    break;
    LASER_GEMV_U(1)
    LASER_GEMV_U(2)
    LASER_GEMV_U(3)
#undef LASER_GEMV_U
  }
  return hipErrorInvalidValue;
}

// Threads of a VALU GEMV workgroup: a.gv_threads, else 256, or 512 for long rows (the down
// projection) so each thread streams fewer chunks.  0: an invalid a.gv_threads.
template <class WT>
static unsigned gemv_threads(const GemmArgs& a, int rw, int rows) {
  if (a.gv_threads > 0) {
    if (a.gv_threads % 64 != 0 || a.gv_threads > kGemvMaxThreads || a.gv_threads < 64 * ((rw * rows + 63) / 64)) return 0;
    return (unsigned)a.gv_threads;
  }
  return a.K / (16 / (int)sizeof(WT)) > 2048 ? kGemvMaxThreads : kGemmThreads;
}

template <class WT, int MODE>
static hipError_t launch_epi(int epi, int rw, const GemmArgs& a, hipStream_t s) {
  const dim3 grid(a.n_groups);
  dim3 block(kGemmThreads);
  if constexpr (MODE <= 4) {
    // chunks in flight per thread: a.gv_u, else 2
    block = dim3(gemv_threads<WT>(a, rw, MODE));
    if (block.x == 0) return hipErrorInvalidValue;
    const int u = a.gv_u > 0 ? a.gv_u : 2;
    switch (epi) {
      case EPI_QKV:
        if (rw == 4) return launch_gemv_u<WT, MODE, EPI_QKV, 4>(u, grid, block, a, s);
        if (rw == 6) return launch_gemv_u<WT, MODE, EPI_QKV, 6>(u, grid, block, a, s);
        if (rw == 8) return launch_gemv_u<WT, MODE, EPI_QKV, 8>(u, grid, block, a, s);
        break;
      case EPI_RESID:
        if (rw == 6) return launch_gemv_u<WT, MODE, EPI_RESID, 6>(u, grid, block, a, s);
        if (rw == 7) return launch_gemv_u<WT, MODE, EPI_RESID, 7>(u, grid, block, a, s);
        if (rw == 8) return launch_gemv_u<WT, MODE, EPI_RESID, 8>(u, grid, block, a, s);
        break;
      case EPI_SWIGLU:
        if (rw == 8) return launch_gemv_u<WT, MODE, EPI_SWIGLU, 8>(u, grid, block, a, s);
        break;
      case EPI_LMHEAD:
        if (rw == 8) return launch_gemv_u<WT, MODE, EPI_LMHEAD, 8>(u, grid, block, a, s);
        break;
    }
    return hipErrorInvalidValue;
  } else {
    constexpr int MT = MODE - 4;
    if (rw != rows_per_group(epi, true)) return hipErrorInvalidValue;
    const int nr = a.nr < 1 ? 1 : a.nr;
    if (!mfma_nr_ok<MT>(nr)) return hipErrorInvalidValue;
    const int ksplit = a.ksplit < 1 ? 1 : a.ksplit;
    if (ksplit > 1 && (epi != EPI_RESID || a.kpart == nullptr || ksplit > kMaxKsplit || a.N % 16 != 0 ||
                       (size_t)ksplit * a.M * a.N * 4 > 0xffffffffu))
      return hipErrorInvalidValue;
    if (a.nrw > 0) {  // row-wave kernel: 8-column activation segments, so K a multiple of 8
      if ((a.nrw != 1 && a.nrw != 2) || a.K % 8 != 0 || a.M < 1 || a.M > 16 * MT) return hipErrorInvalidValue;
      const dim3 grid((a.n_groups + 4 * a.nrw - 1) / (4 * a.nrw) * ksplit);
      return a.nrw == 2 ? launch_mfma_rw<WT, MT, 2>(epi, grid, a, s) : launch_mfma_rw<WT, MT, 1>(epi, grid, a, s);
    }
    const dim3 mgrid((a.n_groups + nr - 1) / nr * ksplit);
    // few workgroups (the O, down and QKV projections): 8 waves split K more finely
    const int waves = mgrid.x < 512 ? kMfmaMaxWaves : kGemmThreads / 64;
    auto blk = [&](int wmax) { return dim3(64 * (waves < wmax ? waves : wmax)); };
    if (nr == 2) return launch_mfma<WT, MT, 2>(epi, mgrid, blk(mfma_wmax<MT, 2>()), a, s);
    if constexpr (mfma_nr_ok<MT>(4)) {
      if (nr == 4) return launch_mfma<WT, MT, 4>(epi, mgrid, blk(mfma_wmax<MT, 4>()), a, s);
    }
    return launch_mfma<WT, MT, 1>(epi, mgrid, blk(mfma_wmax<MT, 1>()), a, s);
  }
}

template <class WT>
static hipError_t launch_mode(int mode, int epi, int rw, const GemmArgs& a, hipStream_t s) {
  switch (mode) {
    case 1: return launch_epi<WT, 1>(epi, rw, a, s);
    case 2: return launch_epi<WT, 2>(epi, rw, a, s);
    case 3: return launch_epi<WT, 3>(epi, rw, a, s);
    case 4: return launch_epi<WT, 4>(epi, rw, a, s);
    case 5: return launch_epi<WT, 5>(epi, rw, a, s);
    case 6: return launch_epi<WT, 6>(epi, rw, a, s);
    case 7: return launch_epi<WT, 7>(epi, rw, a, s);
    case 8: return launch_epi<WT, 8>(epi, rw, a, s);
    default: return hipErrorInvalidValue;
  }
}

template <class WT, int M, int RW>
static hipError_t launch_merged_u(int u, dim3 grid, dim3 block, const GemmArgs& a, const MergeArgs& mg, hipStream_t s) {
  switch (u) {
#define LASER_MERGED_U(UU)                                                           \
  case UU:                                                                           \
    if constexpr (gemv_built<WT, M, EPI_RESID, RW, UU>())                            \
      return launch_k(k_gemv_merged<WT, M, RW, UU>, grid, block, s, a, mg);          \
    break;
    LASER_MERGED_U(1)
    LASER_MERGED_U(2)
    LASER_MERGED_U(3)
#undef LASER_MERGED_U
  }
  return hipErrorInvalidValue;
}

template <class WT, int M>
static hipError_t launch_merged_rw(int rw, const GemmArgs& a, const MergeArgs& mg, hipStream_t s) {
  const dim3 block(gemv_threads<WT>(a, rw, M));
  if (block.x == 0) return hipErrorInvalidValue;
  const dim3 grid(mg.nwg + a.n_groups);
  const int u = a.gv_u > 0 ? a.gv_u : 2;
  if (rw == 6) return launch_merged_u<WT, M, 6>(u, grid, block, a, mg, s);
  if (rw == 7) return launch_merged_u<WT, M, 7>(u, grid, block, a, mg, s);
  if (rw == 8) return launch_merged_u<WT, M, 8>(u, grid, block, a, mg, s);
  return hipErrorInvalidValue;
}

hipError_t launch_gemv_merged(int dtype, int rw, const GemmArgs& a, const MergeArgs& mg, hipStream_t s) {
  if (a.gain != nullptr || a.ksplit > 1 || a.row_map || a.M < 1 || a.M > 2 || mg.nwg != a.M * mg.hq ||
      (mg.hd != 64 && mg.hd != 128) || mg.nslots < 1 || mg.nslots > kAttnMaxWG || mg.cnt == nullptr ||
      a.ldx != mg.hq * mg.hd || (size_t)a.M * a.ldx * 4 > mg.o_bytes || a.K != a.ldx || mg.max_rows < a.M)
    return hipErrorInvalidValue;
  if (dtype == 1) return a.M == 1 ? launch_merged_rw<bf16_t, 1>(rw, a, mg, s) : launch_merged_rw<bf16_t, 2>(rw, a, mg, s);
  return a.M == 1 ? launch_merged_rw<float, 1>(rw, a, mg, s) : launch_merged_rw<float, 2>(rw, a, mg, s);
}

hipError_t launch_gemm(int dtype, int mode, int epi, int rw, const GemmArgs& a, hipStream_t s) {
  if ((a.gain != nullptr) != (epi != EPI_RESID)) return hipErrorInvalidValue;  // only the residual GEMMs skip the norm
  if (mode <= 4 && a.ksplit > 1) return hipErrorInvalidValue;                  // K shares: MFMA path only
  if (dtype == 1) return launch_mode<bf16_t>(mode, epi, rw, a, s);
  return launch_mode<float>(mode, epi, rw, a, s);
}

}  // namespace laser
