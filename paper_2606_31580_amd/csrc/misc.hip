// Small kernels of the forward: embedding gather (+ block-table updates), the LM head's
// softmax merge, KV-cache import/export between the paged layout and a dense one, and the
// probe's confidence mean.
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
__global__ __launch_bounds__(64) void k_embed(const Plan* plan, const void* embed, int d, int vocab, const int* tok0,
                                              const int* tok1, float* h, int* bt, int max_pps) {
  if (blockIdx.x == 0 && blockIdx.y == 0) apply_bt_updates(plan, bt, max_pps);
  const int m = blockIdx.x, g = blockIdx.y, j = threadIdx.x;
  const RowDesc rd = plan->rows[m];
  int tok = (rd.tok_sel == 0 ? tok0 : tok1)[rd.tok_off];
  if (tok < 0 || tok >= vocab) tok = 0;  // ids outside the vocabulary never index past the table
  h[(size_t)m * d + 64 * g + j] = ldw<WT>(embed, (size_t)tok * d + 64 * g + j);
}

// (mx, sum, idx) of a range merged with the statistics of a range of higher indices.
__device__ __forceinline__ void lm_merge(float& mx, float& sum, int& idx, float mx2, float sum2, int idx2) {
  if (mx2 > mx) {
    sum = sum * expf(mx - mx2) + sum2;
    mx = mx2;
    idx = idx2;
  } else if (mx2 == mx) {
    sum += sum2;
  } else {
    sum += sum2 * expf(mx2 - mx);
  }
}

// One workgroup per LM-head output row: merges the per-group softmax statistics in index
// order (contiguous chunks per thread, loaded 8 at a time, then a pairwise tree; ties keep
// the lower index) into the greedy token and p_max = 1 / sum_j exp(l_j - l_max).
constexpr int kLmThreads = 1024;
__global__ __launch_bounds__(kLmThreads) void k_lm_reduce(const Plan* plan, const LmPart* part, int n_groups, int* tok0,
                                                          int* tok1, float* p0, float* p1) {
  __shared__ float s_mx[kLmThreads];
  __shared__ float s_sum[kLmThreads];
  __shared__ int s_idx[kLmThreads];
  const int m = blockIdx.x, tid = threadIdx.x;
  const int C = (n_groups + kLmThreads - 1) / kLmThreads;
  float mx = -INFINITY, sum = 0.f;
  int idx = 0;
  const int g0 = tid * C, g1 = min(g0 + C, n_groups);
  for (int g = g0; g < g1; g += 8) {
    LmPart pp[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (g + u < g1) pp[u] = part[(size_t)(g + u) * kMaxRows + m];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (g + u < g1) lm_merge(mx, sum, idx, pp[u].mx, pp[u].sum, pp[u].idx);
  }
  s_mx[tid] = mx;
  s_sum[tid] = sum;
  s_idx[tid] = idx;
  __syncthreads();
  for (int stride = 1; stride < kLmThreads; stride <<= 1) {
    if ((tid & (2 * stride - 1)) == 0) {
      float m0 = s_mx[tid], su = s_sum[tid];
      int i0 = s_idx[tid];
      lm_merge(m0, su, i0, s_mx[tid + stride], s_sum[tid + stride], s_idx[tid + stride]);
      s_mx[tid] = m0;
      s_sum[tid] = su;
      s_idx[tid] = i0;
    }
    __syncthreads();
  }
  if (tid == 0) {
    const OutDesc od = plan->outs[m];
    (od.sel == 0 ? tok0 : tok1)[od.off] = s_idx[0];
    (od.sel == 0 ? p0 : p1)[od.off] = 1.f / s_sum[0];
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

hipError_t launch_embed(int dtype, const Plan* plan, int M, const void* embed, int d, int vocab, const int* tok0,
                        const int* tok1, float* h, int* bt, int max_pps, hipStream_t s) {
  const dim3 grid(M, d / 64);
  if (dtype == 1)
    hipLaunchKernelGGL(k_embed<bf16_t>, grid, dim3(64), 0, s, plan, embed, d, vocab, tok0, tok1, h, bt, max_pps);
  else
    hipLaunchKernelGGL(k_embed<float>, grid, dim3(64), 0, s, plan, embed, d, vocab, tok0, tok1, h, bt, max_pps);
  return hipGetLastError();
}

hipError_t launch_lm_reduce(const Plan* plan, const LmPart* part, int n_groups, int n_out, int* tok0, int* tok1,
                            float* p0, float* p1, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_reduce, dim3(n_out), dim3(kLmThreads), 0, s, plan, part, n_groups, tok0, tok1, p0, p1);
  return hipGetLastError();
}

hipError_t launch_apply_bt(const Plan* plan, int* bt, int max_pps, hipStream_t s) {
  hipLaunchKernelGGL(k_apply_bt, dim3(1), dim3(256), 0, s, plan, bt, max_pps);
  return hipGetLastError();
}

hipError_t launch_kv_copy(int dtype, int to_pool, void* kpool, void* vpool, const int* bt, int max_pps,
                          int num_pages, int n_layers, int hkv, int hd, int seq, int len, void* k_lin,
                          void* v_lin, hipStream_t s) {
  const size_t total = (size_t)n_layers * len * hkv * hd;
  if (total == 0) return hipSuccess;
  size_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (dtype == 1)
    hipLaunchKernelGGL(k_kv_copy<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, s, to_pool, kpool, vpool, bt,
                       max_pps, num_pages, n_layers, hkv, hd, seq, len, k_lin, v_lin);
  else
    hipLaunchKernelGGL(k_kv_copy<float>, dim3((unsigned)blocks), dim3(256), 0, s, to_pool, kpool, vpool, bt, max_pps,
                       num_pages, n_layers, hkv, hd, seq, len, k_lin, v_lin);
  return hipGetLastError();
}

hipError_t launch_confidence(const float* p, int T, int n, float* conf, hipStream_t s) {
  hipLaunchKernelGGL(k_confidence, dim3((n + 63) / 64), dim3(64), 0, s, p, T, n, conf);
  return hipGetLastError();
}

}  // namespace laser
