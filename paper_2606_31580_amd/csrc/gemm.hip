// Weight-streaming projections of the decoder (the bulk of every decode step's HBM bytes).
//
// One kernel family computes Y = A W^T for A = M activation rows (fp32) and a row-major
// weight matrix W [rows][K] (bf16 or fp32), fused with what precedes and follows it:
//   prologue  RMSNorm of the A rows (gain + sum-of-squares partials from the producer);
//   epilogue  EPI_QKV    bias, rotary embedding of q/k, K/V appended to the paged cache;
//             EPI_RESID  residual add into h plus per-64-column sums of squares of h;
//             EPI_SWIGLU silu(gate) * up;
//             EPI_LMHEAD logits, then a grid-wide merge of (max, sum exp, argmax).
// Work unit = one workgroup = 64 weight rows x one K slice.  Units of the same rows but
// different K slices write fp32 partials; the last unit to arrive (device-scope counter)
// sums them in slice order, so results do not depend on scheduling.
// Main loops:
//   M <= 4  (decode)      VALU: each lane streams 16-byte row-contiguous loads (a wave
//                         instruction reads 1 KB of one row), x from LDS in fp32.
//   M > 4   (probe chunk) MFMA 16x16x32 bf16: weights are the B operand, activations the
//                         A operand split into bf16 hi + lo so the product keeps ~16
//                         significand bits of fp32 activations; fp32 weights are split too.
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

template <class WT, int EPI>
__device__ __forceinline__ const char* weight_row(const GemmArgs& a, int g, int j, bool& valid) {
  const size_t rowbytes = (size_t)a.K * sizeof(WT);
  if (EPI == EPI_QKV) {
    // group g = (head, part): 32 rotary pairs (i, i + hd/2), rows j<32 are the first halves
    const int parts = a.hd >> 6;
    int h = g / parts;
    const int p = g - h * parts;
    const int dim = (j < 32) ? (32 * p + j) : (a.hd / 2 + 32 * p + (j - 32));
    valid = true;
    // h is uniform over the workgroup: pick the matrix with selects, not an indexed lookup
    const bool isq = h < a.hq, isk = !isq && h < a.hq + a.hkv;
    const char* base = (const char*)pick3(isq, isk, a.w0, a.w1, a.w2);
    const int hr = isq ? h : (isk ? h - a.hq : h - a.hq - a.hkv);
    return base + (size_t)(hr * a.hd + dim) * rowbytes;
  } else if (EPI == EPI_SWIGLU) {
    // group g = 32 gate rows and the 32 matching up rows
    int r = 32 * g + (j & 31);
    valid = r < a.F;
    if (!valid) r = 0;
    return (const char*)(j < 32 ? a.w0 : a.w1) + (size_t)r * rowbytes;
  } else {
    int r = 64 * g + j;
    valid = r < a.N;
    if (!valid) r = 0;
    return (const char*)a.w0 + (size_t)r * rowbytes;
  }
}

__device__ __forceinline__ int a_src_row(const GemmArgs& a, int m) { return a.row_map ? a.plan->outs[m].row : m; }


// Stage the unit's slice of the A rows into LDS (fp32, or bf16 hi/lo for MFMA), with the
// RMSNorm prologue applied and zeros past the end of K.
template <class WT, bool MF>
__device__ __forceinline__ void stage_a(const GemmArgs& a, int k0, int klen, int kpad, int M, int ldl, char* smem, float* rms) {
  const int tid = threadIdx.x;
  if (a.gain != nullptr) {
    if (tid < M) {
      const int src = a_src_row(a, tid);
      float s = 0.f;
      for (int gg = 0; gg < a.n_ss; ++gg) s += a.ss[gg * kMaxRows + src];
      rms[tid] = rsqrtf(s / (float)a.K + a.eps);
    }
    __syncthreads();
  }
  for (int idx = tid; idx < M * kpad; idx += blockDim.x) {
    const int m = idx / kpad;
    const int k = idx - m * kpad;
    float v = 0.f;
    if (k < klen) {
      v = a.x[(size_t)a_src_row(a, m) * a.ldx + k0 + k];
      if (a.gain != nullptr) v = v * rms[m] * ldw<WT>(a.gain, (size_t)(k0 + k));
    }
    if (MF) {
      uint16_t hi, lo;
      split_bf16(v, hi, lo);
      uint16_t* xh = (uint16_t*)smem;
      xh[m * ldl + k] = hi;
      xh[M * ldl + m * ldl + k] = lo;
    } else {
      ((float*)smem)[m * ldl + k] = v;
    }
  }
}

// VALU main loop: each wave owns 16 of the unit's 64 rows and streams them R at a time.
template <class WT, int M, int EPI>
__device__ __forceinline__ void valu_main(const GemmArgs& a, int g, int k0, int klen, const float* xs, int ldl, float* Y) {
  constexpr int CH = 16 / (int)sizeof(WT);  // elements per 16-byte load
  constexpr int R = (M == 1) ? 16 : (M == 2 ? 8 : 4);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int nch = klen / CH;
#pragma unroll 1
  for (int pass = 0; pass < 16 / R; ++pass) {
    const char* wp[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      bool valid;
      wp[r] = weight_row<WT, EPI>(a, g, 16 * w + pass * R + r, valid) + (size_t)k0 * sizeof(WT);
    }
    float acc[R][M];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < M; ++m) acc[r][m] = 0.f;
    for (int c = l; c < nch; c += 64) {
      u32x4 v[R];
#pragma unroll
      for (int r = 0; r < R; ++r) v[r] = ld_nt16(wp[r] + (size_t)c * 16);
#pragma unroll
      for (int m = 0; m < M; ++m) {
        float xv[CH];
        const float4* xp = (const float4*)(xs + m * ldl + c * CH);
#pragma unroll
        for (int e4 = 0; e4 < CH / 4; ++e4) {
          float4 t = xp[e4];
          xv[4 * e4 + 0] = t.x;
          xv[4 * e4 + 1] = t.y;
          xv[4 * e4 + 2] = t.z;
          xv[4 * e4 + 3] = t.w;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          float s = acc[r][m];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (sizeof(WT) == 2) {
              s = fmaf(__uint_as_float(v[r][q] << 16), xv[2 * q], s);
              s = fmaf(__uint_as_float(v[r][q] & 0xffff0000u), xv[2 * q + 1], s);
            } else {
              s = fmaf(__uint_as_float(v[r][q]), xv[q], s);
            }
          }
          acc[r][m] = s;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const float s = wave_sum(acc[r][m]);
        if (l == 0) Y[m * 64 + 16 * w + pass * R + r] = s;
      }
  }
}

// MFMA main loop: each wave owns one 16-row n-tile; lane (n, kg) loads 8 consecutive K
// elements of row n; 8 steps of 32 K are kept in flight.
template <class WT, int MT, int EPI>
__device__ __forceinline__ void mfma_main(const GemmArgs& a, int g, int k0, int klen, int M, const uint16_t* xhi,
                          const uint16_t* xlo, int ldl, float* Y) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int n = l & 15, kg = 8 * (l >> 4);
  bool valid;
  const char* wp = weight_row<WT, EPI>(a, g, 16 * w + n, valid) + (size_t)k0 * sizeof(WT);
  const int nsteps = (klen + 31) >> 5;
  int arow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) arow[mt] = min(16 * mt + n, M - 1) * ldl;
  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  constexpr int U = 8;
  constexpr int NLD = (int)sizeof(WT) / 2;  // 16-byte loads per step (bf16: 1, fp32: 2)
  u32x4 buf[U][NLD];
  // 16 bytes q of step s; past the slice any valid row bytes do, the A operand is zero there
  auto ldstep = [&](int s, int q) -> u32x4 {
    int kk = 32 * s + kg;
    if (kk >= klen) kk = 0;
    return ld_nt16(wp + (size_t)kk * sizeof(WT) + 16 * q);
  };
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (u < nsteps)
#pragma unroll
      for (int q = 0; q < NLD; ++q) buf[u][q] = ldstep(u, q);
  for (int s0 = 0; s0 < nsteps; s0 += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + u;
      if (s < nsteps) {
        u32x4 cur[NLD];
#pragma unroll
        for (int q = 0; q < NLD; ++q) cur[q] = buf[u][q];
        if (s + U < nsteps)
#pragma unroll
          for (int q = 0; q < NLD; ++q) buf[u][q] = ldstep(s + U, q);
        const int kk = 32 * s + kg;
        bf16x8 bhi, blo;
        if (NLD == 1) {
          bhi = __builtin_bit_cast(bf16x8, cur[0]);
        } else {
          u32x4 ph, pl;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            uint16_t h0, l0, h1, l1;
            split_bf16(__uint_as_float(cur[q >> 1][(q & 1) * 2 + 0]), h0, l0);
            split_bf16(__uint_as_float(cur[q >> 1][(q & 1) * 2 + 1]), h1, l1);
            ph[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
            pl[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
          }
          bhi = __builtin_bit_cast(bf16x8, ph);
          blo = __builtin_bit_cast(bf16x8, pl);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const bf16x8 ahi = *(const bf16x8*)(xhi + arow[mt] + kk);
          const bf16x8 alo = *(const bf16x8*)(xlo + arow[mt] + kk);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bhi, acc[mt], 0, 0, 0);
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bhi, acc[mt], 0, 0, 0);
          if (NLD == 2) acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, blo, acc[mt], 0, 0, 0);
        }
      }
    }
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 16 * mt + 4 * (l >> 4) + i;
      if (m < M) Y[m * 64 + 16 * w + n] = acc[mt][i];
    }
}

// ----------------------------------------------------------------------------- epilogues

template <class WT>
__device__ __forceinline__ void epi_qkv(const GemmArgs& a, int g, int M, const float* Y) {
  const int parts = a.hd >> 6;
  const int h = g / parts, p = g - h * parts;
  const int half = a.hd >> 1;
  int kind, hh;  // 0: query head, 1: key head, 2: value head
  if (h < a.hq) {
    kind = 0;
    hh = h;
  } else if (h < a.hq + a.hkv) {
    kind = 1;
    hh = h - a.hq;
  } else {
    kind = 2;
    hh = h - a.hq - a.hkv;
  }
  const void* bias = pick3(kind == 0, kind == 1, a.b0, a.b1, a.b2);
  for (int idx = threadIdx.x; idx < M * 32; idx += blockDim.x) {
    const int m = idx >> 5, jj = idx & 31;
    const int i = 32 * p + jj;  // rotary pair index
    const int dlo = i, dhi = half + i;
    float ylo = Y[m * 64 + jj], yhi = Y[m * 64 + 32 + jj];
    if (bias != nullptr) {
      ylo += ldw<WT>(bias, (size_t)hh * a.hd + dlo);
      yhi += ldw<WT>(bias, (size_t)hh * a.hd + dhi);
    }
    const RowDesc rd = a.plan->rows[m];
    if (kind < 2) {
      const float2 cs = a.rope[(size_t)rd.pos * half + i];
      const float rlo = ylo * cs.x - yhi * cs.y;
      const float rhi = yhi * cs.x + ylo * cs.y;
      ylo = rlo;
      yhi = rhi;
    }
    if (kind == 0) {
      float* q = a.q_out + ((size_t)m * a.hq + hh) * a.hd;
      q[dlo] = ylo;
      q[dhi] = yhi;
    } else {
      const int page = a.bt[(size_t)rd.seq * a.max_pps + (rd.pos >> 4)];
      const int t = rd.pos & 15;
      const size_t blk = (((size_t)a.layer * a.num_pages + page) * a.hkv + hh) * (size_t)(16 * a.hd);
      if (kind == 1) {
        stw<WT>(a.kpool, blk + k_block_off(t, dlo), ylo);
        stw<WT>(a.kpool, blk + k_block_off(t, dhi), yhi);
      } else {
        stw<WT>(a.vpool, blk + v_block_off(t, dlo), ylo);
        stw<WT>(a.vpool, blk + v_block_off(t, dhi), yhi);
      }
    }
  }
}

__device__ __forceinline__ void epi_resid(const GemmArgs& a, int g, int M, float* Y) {
  for (int idx = threadIdx.x; idx < M * 64; idx += blockDim.x) {
    const int m = idx >> 6, j = idx & 63;
    const size_t e = (size_t)m * a.N + 64 * g + j;
    const float hv = a.h[e] + Y[idx];
    a.h[e] = hv;
    Y[idx] = hv * hv;
  }
  __syncthreads();
  if ((int)threadIdx.x < M) {
    float s = 0.f;
    for (int j = 0; j < 64; ++j) s += Y[threadIdx.x * 64 + j];
    a.ss_out[g * kMaxRows + threadIdx.x] = s;
  }
}

__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, int g, int M, const float* Y) {
  for (int idx = threadIdx.x; idx < M * 32; idx += blockDim.x) {
    const int m = idx >> 5, jj = idx & 31;
    const int r = 32 * g + jj;
    if (r < a.F) {
      const float gt = Y[m * 64 + jj], up = Y[m * 64 + 32 + jj];
      a.act[(size_t)m * a.F + r] = gt / (1.f + expf(-gt)) * up;
    }
  }
}

// (mx, sum, idx) of a range merged with the stats of a range of higher indices.
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

__device__ __forceinline__ void epi_lmhead(const GemmArgs& a, int g, int M, const float* Y) {
  __shared__ float s_mx[kGemmThreads];
  __shared__ float s_sum[kGemmThreads];
  __shared__ int s_idx[kGemmThreads];
  __shared__ int s_last;
  const int tid = threadIdx.x;
  for (int idx = tid; idx < M * 64; idx += blockDim.x) {
    const int m = idx >> 6, j = idx & 63;
    const int r = 64 * g + j;
    const OutDesc od = a.plan->outs[m];
    if (r < a.N && a.logits[od.sel] != nullptr) a.logits[od.sel][(size_t)od.off * a.N + r] = Y[idx];
  }
  if (tid < M) {
    float mx = -INFINITY;
    int arg = 64 * g;  // a valid id even if no logit compares greater (NaN input)
    for (int j = 0; j < 64; ++j) {
      const int r = 64 * g + j;
      if (r < a.N && Y[tid * 64 + j] > mx) {
        mx = Y[tid * 64 + j];
        arg = r;
      }
    }
    float s = 0.f;
    for (int j = 0; j < 64; ++j) {
      const int r = 64 * g + j;
      if (r < a.N) s += expf(Y[tid * 64 + j] - mx);
    }
    a.lm_part[g * kMaxRows + tid] = LmPart{mx, s, arg, 0};
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) s_last = (atomicAdd(a.lm_cnt, 1) == a.n_groups - 1);
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  // Deterministic merge over all vocabulary groups: contiguous chunks per thread, then a
  // pairwise tree in index order (ties keep the lower index).
  const int C = (a.n_groups + kGemmThreads - 1) / kGemmThreads;
  for (int m = 0; m < M; ++m) {
    float mx = -INFINITY, sum = 0.f;
    int idx = 0;
    const int g0 = tid * C, g1 = min(g0 + C, a.n_groups);
    for (int gg = g0; gg < g1; ++gg) {
      const LmPart pp = a.lm_part[gg * kMaxRows + m];
      lm_merge(mx, sum, idx, pp.mx, pp.sum, pp.idx);
    }
    s_mx[tid] = mx;
    s_sum[tid] = sum;
    s_idx[tid] = idx;
    __syncthreads();
    for (int stride = 1; stride < kGemmThreads; stride <<= 1) {
      if ((tid & (2 * stride - 1)) == 0 && tid + stride < kGemmThreads) {
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
      const OutDesc od = a.plan->outs[m];
      a.tok_out[od.sel][od.off] = s_idx[0];
      a.p_out[od.sel][od.off] = 1.f / s_sum[0];
    }
    __syncthreads();
  }
  if (tid == 0) *a.lm_cnt = 0;
}

// ----------------------------------------------------------------------------- kernel

template <class WT, int MODE, int EPI>
__global__ __launch_bounds__(kGemmThreads) void k_gemm(GemmArgs a) {
  extern __shared__ __align__(16) char smem[];
  __shared__ float s_rms[kMaxRows];
  __shared__ int s_last;
  constexpr bool MF = MODE > 4;
  const int unit = blockIdx.x;
  const int g = unit / a.n_splits, sp = unit - g * a.n_splits;
  const int k0 = sp * a.kslice;
  const int klen = min(a.kslice, a.K - k0);
  const int M = a.M;
  int ldl, kpad, stage_bytes;
  if (MF) {
    ldl = ((a.kslice + 31) & ~31) + 8;
    kpad = (klen + 31) & ~31;
    stage_bytes = 4 * M * ldl;
  } else {
    ldl = a.kslice;
    kpad = klen;
    stage_bytes = 4 * M * ldl;
  }
  float* Y = (float*)(smem + stage_bytes);
  stage_a<WT, MF>(a, k0, klen, kpad, M, ldl, smem, s_rms);
  __syncthreads();
  if (MF) {
    const uint16_t* xh = (const uint16_t*)smem;
    mfma_main<WT, (MF ? MODE - 4 : 1), EPI>(a, g, k0, klen, M, xh, xh + M * ldl, ldl, Y);
  } else {
    valu_main<WT, (MF ? 1 : MODE), EPI>(a, g, k0, klen, (const float*)smem, ldl, Y);
  }
  __syncthreads();
  if (a.n_splits > 1) {
    float* mine = a.part + (size_t)(g * a.n_splits + sp) * M * 64;
    for (int idx = threadIdx.x; idx < M * 64; idx += blockDim.x) mine[idx] = Y[idx];
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) s_last = (atomicAdd(&a.cnt[g], 1) == a.n_splits - 1);
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const float* base = a.part + (size_t)g * a.n_splits * M * 64;
    for (int idx = threadIdx.x; idx < M * 64; idx += blockDim.x) {
      float s = 0.f;
      for (int q = 0; q < a.n_splits; ++q) s += __builtin_nontemporal_load(base + (size_t)q * M * 64 + idx);
      Y[idx] = s;
    }
    if (threadIdx.x == 0) a.cnt[g] = 0;
    __syncthreads();
  }
  if (EPI == EPI_QKV) epi_qkv<WT>(a, g, M, Y);
  if (EPI == EPI_RESID) epi_resid(a, g, M, Y);
  if (EPI == EPI_SWIGLU) epi_swiglu(a, g, M, Y);
  if (EPI == EPI_LMHEAD) epi_lmhead(a, g, M, Y);
}

size_t gemm_lds_bytes(int dtype, int mode, int kslice, int M) {
  (void)dtype;
  const int ldl = mode > 4 ? ((kslice + 31) & ~31) + 8 : kslice;
  return (size_t)4 * M * ldl + (size_t)4 * M * 64;
}

template <class WT, int MODE>
static hipError_t launch_epi(int epi, const GemmArgs& a, int grid, size_t lds, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: hipLaunchKernelGGL((k_gemm<WT, MODE, EPI_QKV>), dim3(grid), dim3(kGemmThreads), lds, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((k_gemm<WT, MODE, EPI_RESID>), dim3(grid), dim3(kGemmThreads), lds, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((k_gemm<WT, MODE, EPI_SWIGLU>), dim3(grid), dim3(kGemmThreads), lds, s, a); break;
    case EPI_LMHEAD: hipLaunchKernelGGL((k_gemm<WT, MODE, EPI_LMHEAD>), dim3(grid), dim3(kGemmThreads), lds, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class WT>
static hipError_t launch_mode(int mode, int epi, const GemmArgs& a, int grid, size_t lds, hipStream_t s) {
  switch (mode) {
    case 1: return launch_epi<WT, 1>(epi, a, grid, lds, s);
    case 2: return launch_epi<WT, 2>(epi, a, grid, lds, s);
    case 3: return launch_epi<WT, 3>(epi, a, grid, lds, s);
    case 4: return launch_epi<WT, 4>(epi, a, grid, lds, s);
    case 5: return launch_epi<WT, 5>(epi, a, grid, lds, s);
    case 6: return launch_epi<WT, 6>(epi, a, grid, lds, s);
    case 7: return launch_epi<WT, 7>(epi, a, grid, lds, s);
    case 8: return launch_epi<WT, 8>(epi, a, grid, lds, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(int dtype, int mode, int epi, const GemmArgs& a, int grid, hipStream_t s) {
  const size_t lds = gemm_lds_bytes(dtype, mode, a.kslice, a.M);
  if (dtype == 1) return launch_mode<bf16_t>(mode, epi, a, grid, lds, s);
  return launch_mode<float>(mode, epi, a, grid, lds, s);
}

}  // namespace laser
