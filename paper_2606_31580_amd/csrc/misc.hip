// Small kernels of the forward: embedding gather (+ block-table updates), the LM head's
// softmax merge, KV-cache import/export between the paged layout and a dense one, and the
// probe's confidence mean.
#include <algorithm>
#include <cstddef>

#include "device_common.hpp"
#include "kernels.hpp"

namespace laser {

__device__ void apply_bt_updates(const Plan* plan, int* bt, int max_pps) {
  for (int i = threadIdx.x; i < plan->n_bt; i += blockDim.x) {
    const BtUpdate u = plan->bt[i];
    bt[(size_t)u.seq * max_pps + u.idx] = u.page;
  }
}

// grid (M, d/64), block 64: h[m][64g..64g+63] = embed[token(m)].
template <class WT>
__global__ __launch_bounds__(64) void k_embed(const Plan* plan, const void* embed, int d, int vocab, float* h, int* bt,
                                              int max_pps) {
  if (blockIdx.x == 0 && blockIdx.y == 0) apply_bt_updates(plan, bt, max_pps);
  const int m = blockIdx.x, g = blockIdx.y, j = threadIdx.x;
  const RowDesc rd = plan->rows[m];
  int tok = plan->io.tok_src[rd.tok_sel][rd.tok_off];
  if (tok < 0 || tok >= vocab) tok = 0;  // ids outside the vocabulary never index past the table
  h[(size_t)m * d + 64 * g + j] = ldw<WT>(embed, (size_t)tok * d + 64 * g + j);
}

// One workgroup per LM-head output row: merges the per-group softmax statistics into the
// greedy token (lowest index among equal maxima) and p_max = 1 / sum_j exp(l_j - l_max).
// Every thread loads all its groups at once (a 152k vocabulary at 8 rows per group is one
// round), then the maximum is reduced first (lanes, waves) and the sums are rescaled to it
// once, so no merge step needs an exponential of its own.  Indices are exact as floats
// (below 2^24), which lets the lowest index be a plain minimum reduction.
constexpr int kLmThreads = 1024;
constexpr int kLmPer = 20;  // groups per thread per round
__global__ __launch_bounds__(kLmThreads) void k_lm_reduce(const Plan* plan, const LmPart* part, int n_groups) {
  constexpr int NW = kLmThreads / 64;
  constexpr float kNoIdx = 3.0e38f;
  __shared__ float s_mx[NW], s_sum[NW], s_idx[NW];
  const int m = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const LmPart* row = part + (size_t)m * n_groups;
  float mx = -INFINITY, sum = 0.f, idx = kNoIdx;
  for (int g0 = tid; g0 < n_groups; g0 += kLmPer * kLmThreads) {
    LmPart pp[kLmPer];
#pragma unroll
    for (int u = 0; u < kLmPer; ++u) {
      const int g = g0 + u * kLmThreads;
      pp[u] = g < n_groups ? row[g] : LmPart{-INFINITY, 0.f, 0x7fffffff, 0};
    }
    float rm = mx;
#pragma unroll
    for (int u = 0; u < kLmPer; ++u) rm = fmaxf(rm, pp[u].mx);
    float rs = (mx == rm) ? sum : (mx == -INFINITY ? 0.f : sum * expf(mx - rm));
    float ri = (mx == rm) ? idx : kNoIdx;
#pragma unroll
    for (int u = 0; u < kLmPer; ++u) {
      if (pp[u].mx == rm) {
        rs += pp[u].sum;
        if (pp[u].idx != 0x7fffffff) ri = fminf(ri, (float)pp[u].idx);
      } else if (pp[u].mx != -INFINITY) {
        rs += pp[u].sum * expf(pp[u].mx - rm);
      }
    }
    mx = rm;
    sum = rs;
    idx = ri;
  }
  // maximum over the workgroup
  const float wm = wave_max(mx);
  if (lane == 0) s_mx[w] = wm;
  __syncthreads();
  float M = s_mx[0];
#pragma unroll
  for (int v = 1; v < NW; ++v) M = fmaxf(M, s_mx[v]);
  // sums rescaled to it; lowest index among the lanes at it
  const float mine = (mx == -INFINITY || M == -INFINITY) ? 0.f : (mx == M ? sum : sum * expf(mx - M));
  const float ws = wave_sum(mine);
  const float wi = wave_min(mx == M ? idx : kNoIdx);
  if (lane == 0) {
    s_sum[w] = ws;
    s_idx[w] = wi;
  }
  __syncthreads();
  if (tid == 0) {
    float tot = 0.f, best = kNoIdx;
    for (int v = 0; v < NW; ++v) {  // fixed order
      tot += s_sum[v];
      best = fminf(best, s_idx[v]);
    }
    const OutDesc od = plan->outs[m];
    plan->io.tok_dst[od.sel][od.off] = best >= kNoIdx ? 0 : (int)best;
    plan->io.p_dst[od.sel][od.off] = 1.f / tot;
  }
}

__global__ void k_apply_bt(const Plan* plan, int* bt, int max_pps) { apply_bt_updates(plan, bt, max_pps); }

// Copy one sequence between the paged pools and dense [n_layers][len][hkv][hd] arrays.
template <class WT>
__global__ void k_kv_copy(int to_pool, void* kpool, void* vpool, const int* bt, int max_pps, int num_pages,
                          int n_layers, int hkv, int hd, int seq, int len, void* k_lin, void* v_lin) {
  const size_t total = (size_t)n_layers * len * hkv * hd;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += stride) {
    const int d = (int)(e % hd);
    size_t r = e / hd;
    const int kvh = (int)(r % hkv);
    r /= hkv;
    const int pos = (int)(r % len);
    const int layer = (int)(r / len);
    const int page = bt[(size_t)seq * max_pps + (pos >> 4)];
    const size_t blk = (((size_t)layer * num_pages + page) * hkv + kvh) * (size_t)(16 * hd);
    const size_t ko = blk + k_block_off(pos & 15, d), vo = blk + v_block_off(pos & 15, d);
    if (to_pool) {
      ((WT*)kpool)[ko] = ((const WT*)k_lin)[e];
      ((WT*)vpool)[vo] = ((const WT*)v_lin)[e];
    } else {
      ((WT*)k_lin)[e] = ((const WT*)kpool)[ko];
      ((WT*)v_lin)[e] = ((const WT*)vpool)[vo];
    }
  }
}

// conf[r] = (p[r*T] + ... + p[r*T + T-1]) / T, summed in trial order.
__global__ void k_confidence(const float* p, int T, int n, float* conf) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  float s = 0.f;
  for (int j = 0; j < T; ++j) s += p[r * T + j];
  conf[r] = s / (float)T;
}

// ATP cue detection: flags[i] = membership of tokens[i] in the bitmap set.
__global__ void k_atp_match(const int* tokens, int n, const unsigned* bitmap, int vocab, int* flags) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int t = tokens[i];
  flags[i] = (t >= 0 && t < vocab) ? (int)((bitmap[t >> 5] >> (t & 31)) & 1u) : 0;
}

// Copy of one page (every layer and kv head, K and V) from page src to page dst: grid
// (n_layers * hkv), 16-byte chunks of the 16 x hd block.
__global__ __launch_bounds__(256) void k_page_copy(void* kpool, void* vpool, int num_pages, int hkv, size_t blk_bytes,
                                                   int src, int dst) {
  const int layer = blockIdx.x / hkv, h = blockIdx.x - layer * hkv;
  const size_t s_off = (((size_t)layer * num_pages + src) * hkv + h) * blk_bytes;
  const size_t d_off = (((size_t)layer * num_pages + dst) * hkv + h) * blk_bytes;
  for (size_t c = threadIdx.x; c < blk_bytes / 16; c += blockDim.x) {
    *(u32x4*)((char*)kpool + d_off + 16 * c) = *(const u32x4*)((const char*)kpool + s_off + 16 * c);
    *(u32x4*)((char*)vpool + d_off + 16 * c) = *(const u32x4*)((const char*)vpool + s_off + 16 * c);
  }
}

hipError_t launch_page_copy(int kv_es, void* kpool, void* vpool, int num_pages, int n_layers, int hkv, int hd, int src,
                            int dst, hipStream_t s) {
  const size_t blk_bytes = (size_t)16 * hd * kv_es;
  return launch_k(k_page_copy, dim3(n_layers * hkv), dim3(256), s, kpool, vpool, num_pages, hkv, blk_bytes, src, dst);
}

hipError_t launch_embed(int dtype, const Plan* plan, int M, const void* embed, int d, int vocab, float* h, int* bt,
                        int max_pps, hipStream_t s) {
  const dim3 grid(M, d / 64);
  if (dtype == 1)
    return launch_k(k_embed<bf16_t>, grid, dim3(64), s, plan, embed, d, vocab, h, bt, max_pps);
  else
    return launch_k(k_embed<float>, grid, dim3(64), s, plan, embed, d, vocab, h, bt, max_pps);
}

hipError_t launch_lm_reduce(const Plan* plan, const LmPart* part, int n_groups, int n_out, hipStream_t s) {
  return launch_k(k_lm_reduce, dim3(n_out), dim3(kLmThreads), s, plan, part, n_groups);
}

// Copies the used part of a plan from its pinned host staging slot (fine-grained memory, read
// over the bus) to the device plan slot: the fixed head and the first work items in one round
// of loads (16 KB), then the rest of the items and the block-table updates, whose counts the
// head gives.  One workgroup; the next kernel of the forward sees the copy after the boundary.
constexpr int kFetchThreads = 1024;
__global__ __launch_bounds__(kFetchThreads) void k_plan_fetch(const Plan* src, Plan* dst) {
  const char* s = (const char*)src;
  char* d = (char*)dst;
  const int t = threadIdx.x;
  __shared__ int s_cnt[2];
  constexpr size_t R1 = 16 * kFetchThreads;
  static_assert(offsetof(Plan, n_items) < 32 && offsetof(Plan, n_bt) < 16, "counts in the first two chunks");
  static_assert(R1 <= offsetof(Plan, bt), "the first round stays inside the head and items");
  const u32x4 v = ld_global<u32x4>(s + 16 * t);
  *(u32x4*)(d + 16 * t) = v;
  if (t == 0) s_cnt[0] = (int)v[offsetof(Plan, n_bt) / 4];
  if (t == 1) s_cnt[1] = (int)v[(offsetof(Plan, n_items) - 16) / 4];
  __syncthreads();
  const int n_bt = min(max(s_cnt[0], 0), kMaxBt), n_items = min(max(s_cnt[1], 0), kMaxAttnItems);
  const size_t items_end = (offsetof(Plan, items) + sizeof(AttnItem) * (size_t)n_items + 15) & ~(size_t)15;
  for (size_t o = R1 + 16 * t; o < items_end; o += 4 * 16 * kFetchThreads) {
    u32x4 w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const size_t ou = o + (size_t)u * 16 * kFetchThreads;
      w[u] = ld_global<u32x4>(s + (ou < items_end ? ou : o));
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const size_t ou = o + (size_t)u * 16 * kFetchThreads;
      if (ou < items_end) *(u32x4*)(d + ou) = w[u];
    }
  }
  // block-table updates: 12-byte entries from a 16-byte aligned start, whole chunks
  static_assert(offsetof(Plan, bt) % 16 == 0, "block-table updates 16-byte aligned");
  const size_t bt_end = offsetof(Plan, bt) + ((sizeof(BtUpdate) * (size_t)n_bt + 15) & ~(size_t)15);
  for (size_t o = offsetof(Plan, bt) + 16 * t; o < bt_end; o += 16 * kFetchThreads)
    *(u32x4*)(d + o) = ld_global<u32x4>(s + o);
}

hipError_t launch_plan_fetch(const Plan* src, Plan* dst, hipStream_t s) {
  return launch_k(k_plan_fetch, dim3(1), dim3(kFetchThreads), s, src, dst);
}

const void* plan_fetch_kernel() { return reinterpret_cast<const void*>(&k_plan_fetch); }

hipError_t launch_apply_bt(const Plan* plan, int* bt, int max_pps, hipStream_t s) {
  hipLaunchKernelGGL(k_apply_bt, dim3(1), dim3(256), 0, s, plan, bt, max_pps);
  return hipGetLastError();
}

hipError_t launch_kv_copy(int kv_es, int to_pool, void* kpool, void* vpool, const int* bt, int max_pps,
                          int num_pages, int n_layers, int hkv, int hd, int seq, int len, void* k_lin,
                          void* v_lin, hipStream_t s) {
  const size_t total = (size_t)n_layers * len * hkv * hd;
  if (total == 0) return hipSuccess;
  size_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (kv_es == 1)
    hipLaunchKernelGGL(k_kv_copy<uint8_t>, dim3((unsigned)blocks), dim3(256), 0, s, to_pool, kpool, vpool, bt,
                       max_pps, num_pages, n_layers, hkv, hd, seq, len, k_lin, v_lin);
  else if (kv_es == 2)
    hipLaunchKernelGGL(k_kv_copy<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, s, to_pool, kpool, vpool, bt,
                       max_pps, num_pages, n_layers, hkv, hd, seq, len, k_lin, v_lin);
  else
    hipLaunchKernelGGL(k_kv_copy<float>, dim3((unsigned)blocks), dim3(256), 0, s, to_pool, kpool, vpool, bt, max_pps,
                       num_pages, n_layers, hkv, hd, seq, len, k_lin, v_lin);
  return hipGetLastError();
}

// p[0 .. n-1] = v (a kernel rather than a memset, so that a caller may capture it in a graph).
__global__ void k_fill_u32(unsigned* p, int n, unsigned v) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = v;
}

hipError_t launch_fill_u32(unsigned* p, int n, unsigned v, hipStream_t s) {
  if (n < 1) return hipSuccess;
  return launch_k(k_fill_u32, dim3(std::min((n + 255) / 256, 1024)), dim3(256), s, p, n, v);
}

hipError_t launch_confidence(const float* p, int T, int n, float* conf, hipStream_t s) {
  return launch_k(k_confidence, dim3((n + 63) / 64), dim3(64), s, p, T, n, conf);
}

hipError_t launch_atp_match(const int* tokens, int n, const unsigned* bitmap, int vocab, int* flags, hipStream_t s) {
  return launch_k(k_atp_match, dim3((n + 255) / 256), dim3(256), s, tokens, n, bitmap, vocab, flags);
}

}  // namespace laser
