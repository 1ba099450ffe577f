// Small kernels of the forward: embedding gather (+ block-table updates), KV-cache
// import/export between the paged layout and a dense one, and the probe's confidence mean.
#include "device_common.hpp"
#include "kernels.hpp"

namespace laser {

__device__ void apply_bt_updates(const Plan* plan, int* bt, int max_pps) {
  for (int i = threadIdx.x; i < plan->n_bt; i += blockDim.x) {
    const BtUpdate u = plan->bt[i];
    bt[(size_t)u.seq * max_pps + u.idx] = u.page;
  }
}

// grid (M, d/64), block 64: h[m][64g..64g+63] = embed[token(m)] and its sum of squares.
template <class WT>
__global__ __launch_bounds__(64) void k_embed(const Plan* plan, const void* embed, int d, int vocab, const int* tok0,
                                              const int* tok1, float* h, float* ss, int* bt, int max_pps) {
  if (blockIdx.x == 0 && blockIdx.y == 0) apply_bt_updates(plan, bt, max_pps);
  const int m = blockIdx.x, g = blockIdx.y, j = threadIdx.x;
  const RowDesc rd = plan->rows[m];
  int tok = (rd.tok_sel == 0 ? tok0 : tok1)[rd.tok_off];
  if (tok < 0 || tok >= vocab) tok = 0;  // ids outside the vocabulary never index past the table
  const float v = ldw<WT>(embed, (size_t)tok * d + 64 * g + j);
  h[(size_t)m * d + 64 * g + j] = v;
  __shared__ float sq[64];
  sq[j] = v * v;
  __syncthreads();
  if (j == 0) {
    float s = 0.f;
    for (int q = 0; q < 64; ++q) s += sq[q];
    ss[g * kMaxRows + m] = s;
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
                        const int* tok1, float* h, float* ss, int* bt, int max_pps, hipStream_t s) {
  const dim3 grid(M, d / 64);
  if (dtype == 1)
    hipLaunchKernelGGL(k_embed<bf16_t>, grid, dim3(64), 0, s, plan, embed, d, vocab, tok0, tok1, h, ss, bt, max_pps);
  else
    hipLaunchKernelGGL(k_embed<float>, grid, dim3(64), 0, s, plan, embed, d, vocab, tok0, tok1, h, ss, bt, max_pps);
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
