// Measurements behind the kernel structure of the decode step (run by `bench.py --design-probes`):
//   1. streaming read: a plain weight-streaming read at several sizes (time = a + bytes / BW);
//   2. kernel boundary: a graph of back-to-back empty kernels;
//   3. cross-workgroup hand-off: every workgroup publishes a row and bumps a counter, the last
//      one reads every row back -- with plain stores, with agent-scope fences, with
//      device-scope (sc1) buffer stores and loads -- counting stale reads;
//   4. grid barrier: cooperative launch, every workgroup resident, bounded spins (a workgroup
//      that waits too long raises a flag and stops), one counter or two levels;
//   5. two dependent weight-streaming products shaped like the 7B gate/up (271.6 MB) and down
//      (135.8 MB) projections: two kernels, or one launch whose second-stage workgroups
//      (dispatched after every first-stage one) load their first weights, wait for a
//      completion counter (bounded spin) and read the first stage's output;
//   6. memory-side cache: a region streamed right after another kernel read it (plain or
//      non-temporal loads), against the same region cold (after a 1 GiB read of other data).
// Every access is in bounds and every wait is bounded.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <vector>

#define CK(x)                                                                            \
  do {                                                                                   \
    hipError_t ck_e_ = (x);                                                              \
    if (ck_e_ != hipSuccess) {                                                           \
      printf("%s: %s\n", #x, hipGetErrorString(ck_e_));                                  \
      exit(1);                                                                           \
    }                                                                                    \
  } while (0)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int TPB = 256;
constexpr unsigned kSpinCap = 1u << 22;

__device__ __forceinline__ void wait_mem() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ f32x4 ld_dev16(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 16));
}
__device__ __forceinline__ u32x4 ldnt(const void* p) { return __builtin_nontemporal_load((const u32x4*)p); }

static float time_ms(hipEvent_t a, hipEvent_t b) {
  float ms = 0.f;
  CK(hipEventElapsedTime(&ms, a, b));
  return ms;
}

// ---------------------------------------------------------------- 1. streaming read
__global__ __launch_bounds__(TPB) void k_stream(const u32x4* p, size_t n16, unsigned* sink) {
  unsigned acc = 0;
  for (size_t i = (size_t)blockIdx.x * TPB + threadIdx.x; i < n16; i += (size_t)gridDim.x * TPB) {
    const u32x4 v = ldnt(p + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == 0x9e3779b9u) sink[0] = acc;  // (keeps the loads)
}

static void stream_read() {
  printf("## 1. streaming read (non-temporal 16-byte loads, 2048 workgroups of 256 threads)\n");
  printf("(each launch reads the next region of a 4 GiB buffer, so nothing is served from the\n"
         " 256 MB memory-side cache of an earlier launch)\n");
  const size_t pool = (size_t)4 << 30;
  u32x4* p;
  unsigned* sink;
  CK(hipMalloc(&p, pool));
  CK(hipMalloc(&sink, 64));
  CK(hipMemset(p, 1, pool));
  hipEvent_t a, b;
  CK(hipEventCreate(&a));
  CK(hipEventCreate(&b));
  std::vector<double> xs, ys;
  for (size_t mb : {16, 32, 64, 128, 256, 512, 1024}) {
    const size_t bytes = mb << 20, n16 = bytes / 16, regions = pool / bytes;
    for (int i = 0; i < 3; ++i) k_stream<<<2048, TPB>>>(p + (i % regions) * n16, n16, sink);
    CK(hipDeviceSynchronize());
    const int reps = 20;
    CK(hipEventRecord(a));
    for (int i = 0; i < reps; ++i) k_stream<<<2048, TPB>>>(p + ((3 + i) % regions) * n16, n16, sink);
    CK(hipEventRecord(b));
    CK(hipDeviceSynchronize());
    const double us = time_ms(a, b) * 1e3 / reps;
    printf("%5zu MiB: %8.2f us, %6.0f GB/s\n", mb, us, bytes / us / 1e3);
    xs.push_back((double)bytes);
    ys.push_back(us);
  }
  double sx = 0, sy = 0, sxx = 0, sxy = 0;  // least-squares fit t = a + bytes / BW
  const int n = (int)xs.size();
  for (int i = 0; i < n; ++i) {
    sx += xs[i];
    sy += ys[i];
    sxx += xs[i] * xs[i];
    sxy += xs[i] * ys[i];
  }
  const double slope = (n * sxy - sx * sy) / (n * sxx - sx * sx), icpt = (sy - slope * sx) / n;
  printf("fit: t = %.2f us + bytes / %.0f GB/s\n\n", icpt, 1e-3 / slope);
  CK(hipFree(p));
  CK(hipFree(sink));
}

// ---------------------------------------------------------------- 2. kernel boundary
__global__ void k_empty(float* p) {
  if (threadIdx.x == 0 && blockIdx.x == 0 && p[0] == 12345.f) p[1] = 1.f;
}

static void graph_boundary() {
  printf("## 2. kernel boundary (graph of 200 back-to-back empty kernels)\n");
  float* p;
  CK(hipMalloc(&p, 64));
  CK(hipMemset(p, 0, 64));
  hipStream_t s;
  CK(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));
  for (int N : {512, 2048}) {
    hipGraph_t g;
    hipGraphExec_t ge;
    CK(hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal));
    for (int i = 0; i < 200; ++i) k_empty<<<N, TPB, 0, s>>>(p);
    CK(hipStreamEndCapture(s, &g));
    CK(hipGraphInstantiate(&ge, g, nullptr, nullptr, 0));
    CK(hipGraphLaunch(ge, s));
    CK(hipStreamSynchronize(s));
    hipEvent_t a, b;
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
    CK(hipEventRecord(a, s));
    CK(hipGraphLaunch(ge, s));
    CK(hipEventRecord(b, s));
    CK(hipStreamSynchronize(s));
    printf("%4d workgroups: %.2f us per kernel\n", N, time_ms(a, b) * 1e3 / 200);
    CK(hipGraphExecDestroy(ge));
    CK(hipGraphDestroy(g));
  }
  printf("\n");
  CK(hipStreamDestroy(s));
  CK(hipFree(p));
}

// ---------------------------------------------------------------- 3. hand-off
// mode 0: plain stores; 1: agent-scope release fence before the counter, acquire fence in the
// last workgroup; 2: device-scope stores, wait, counter, device-scope loads in the last.
template <int MODE>
__global__ __launch_bounds__(TPB) void k_publish(float* data, unsigned* cnt, unsigned* err, float val) {
  const int wg = blockIdx.x, t = threadIdx.x;
  if (MODE == 2)
    __hip_atomic_store(data + (size_t)wg * TPB + t, val, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    data[(size_t)wg * TPB + t] = val;
  if (MODE == 1) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  if (MODE == 2) wait_mem();
  __shared__ unsigned s_t;
  __syncthreads();
  if (t == 0) s_t = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_t != gridDim.x - 1) return;
  if (MODE == 1) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  unsigned bad = 0;
  for (int w = t; w < (int)gridDim.x; w += TPB) {  // element w % TPB of every workgroup
    const size_t i = (size_t)w * TPB + (w % TPB);
    const float x = MODE == 1 ? data[i] : __hip_atomic_load(data + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bad += x != val;
  }
  if (bad) atomicAdd(err, bad);
  if (t == 0) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int MODE>
static void publish(int N, float* data, unsigned* cnt, unsigned* err) {
  CK(hipMemset(cnt, 0, 4));
  CK(hipMemset(err, 0, 4));
  hipEvent_t a, b;
  CK(hipEventCreate(&a));
  CK(hipEventCreate(&b));
  for (int i = 0; i < 10; ++i) k_publish<MODE><<<N, TPB>>>(data, cnt, err, (float)(1000 + i));
  CK(hipDeviceSynchronize());
  const int reps = 200;
  CK(hipEventRecord(a));
  for (int i = 0; i < reps; ++i) k_publish<MODE><<<N, TPB>>>(data, cnt, err, (float)(i + 1));
  CK(hipEventRecord(b));
  CK(hipDeviceSynchronize());
  unsigned e = 0;
  CK(hipMemcpy(&e, err, 4, hipMemcpyDeviceToHost));
  static const char* names[] = {"plain stores", "agent fences", "device-scope stores/loads"};
  printf("%-26s %4d workgroups: %6.2f us per launch (back to back), stale reads %u\n", names[MODE], N,
         time_ms(a, b) * 1e3 / reps, e);
}

// ---------------------------------------------------------------- 4. grid barrier
template <bool TWO>
__global__ __launch_bounds__(TPB) void k_barrier(float* slot, unsigned* cnt, unsigned* err, unsigned* fail, int R) {
  const int wg = blockIdx.x, t = threadIdx.x, N = gridDim.x;
  constexpr int GS = 16;
  const int ng = (N + GS - 1) / GS, grp = wg / GS, gsize = min(GS, N - grp * GS);
  __shared__ int s_ok;
  for (int r = 0; r < R; ++r) {
    if (t == 0) {
      __hip_atomic_store(slot + wg, (float)(r + 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      wait_mem();
      unsigned* flag;
      unsigned target;
      if (TWO) {  // group counter, then the group's last bumps the top; the last group releases
        const unsigned g = __hip_atomic_fetch_add(cnt + 64 * (1 + grp), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (g == (unsigned)gsize * (r + 1) - 1) {
          const unsigned tt = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (tt == (unsigned)ng * (r + 1) - 1)
            for (int k = 0; k < ng; ++k)
              __hip_atomic_store(cnt + 64 * (1 + ng + k), (unsigned)(r + 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        flag = cnt + 64 * (1 + ng + grp);
        target = (unsigned)(r + 1);
      } else {
        __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        flag = cnt;
        target = (unsigned)N * (r + 1);
      }
      unsigned spins = 0;
      int ok = 1;
      while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinCap) {
          ok = 0;
          break;
        }
      }
      if (!ok) atomicOr(fail, 1u);
      s_ok = ok;
    }
    __syncthreads();
    if (!s_ok) return;
    if (t == 0) {
      const int o = (wg + 37) % N;
      if (__hip_atomic_load(slot + o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < (float)(r + 1)) atomicAdd(err, 1u);
    }
    __syncthreads();
  }
}

template <bool TWO>
static void barrier(int N, float* slot, unsigned* cnt, unsigned* err, unsigned* fail) {
  int per_cu = 0, cus = 0;
  CK(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_barrier<TWO>, TPB, 0));
  CK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
  if (N > per_cu * cus) {
    printf("barrier: %d workgroups exceed the resident %d\n", N, per_cu * cus);
    return;
  }
  int R = 200;
  for (int pass = 0; pass < 2; ++pass) {  // (the first launch pays the kernel's first load)
    CK(hipMemset(cnt, 0, 64 * 4 * 80));
    CK(hipMemset(err, 0, 4));
    CK(hipMemset(fail, 0, 4));
    CK(hipMemset(slot, 0, 4 * N));
    hipEvent_t a, b;
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
    void* args[] = {&slot, &cnt, &err, &fail, &R};
    CK(hipEventRecord(a));
    CK(hipLaunchCooperativeKernel((void*)k_barrier<TWO>, dim3(N), dim3(TPB), args, 0, 0));
    CK(hipEventRecord(b));
    CK(hipDeviceSynchronize());
    unsigned e = 0, f = 0;
    CK(hipMemcpy(&e, err, 4, hipMemcpyDeviceToHost));
    CK(hipMemcpy(&f, fail, 4, hipMemcpyDeviceToHost));
    if (pass == 1)
      printf("%-10s %4d workgroups: %5.2f us per barrier over %d rounds, stale reads %u, gave up %u\n",
             TWO ? "two-level" : "one counter", N, time_ms(a, b) * 1e3 / R, R, e, f);
  }
}

// ---------------------------------------------------------------- 5. dependent products
constexpr int U = 2, NCNT = 64;

// RW rows [row0, row0 + RW) of W [rows][K] (bf16) times x (fp32 [K]) into y (dev: device-scope
// stores).  wpre: the first pass's weights, loaded by the caller.  XDEV: x read with
// device-scope loads.
template <int RW, bool XDEV>
__device__ void gemv_rows(const uint16_t* W, int K, const float* x, int row0, int rows, float* y, bool ydev,
                          const u32x4 (*wpre)[RW]) {
  __shared__ float red[TPB / 64][RW];
  const int tid = threadIdx.x, nch = K / 8;
  const __amdgpu_buffer_rsrc_t rx = rsrc(x, (unsigned)K * 4);
  float acc[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) acc[r] = 0.f;
  for (int c0 = tid, pass = 0; c0 < nch; c0 += U * TPB, ++pass) {
    u32x4 wv[U][RW];
    f32x4 xv[U][2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = min(c0 + u * TPB, nch - 1);
#pragma unroll
      for (int r = 0; r < RW; ++r)
        wv[u][r] = (pass == 0 && wpre) ? wpre[u][r] : ldnt(W + (size_t)min(row0 + r, rows - 1) * K + c * 8);
#pragma unroll
      for (int e = 0; e < 2; ++e)
        xv[u][e] = XDEV ? ld_dev16(rx, (unsigned)((c * 8 + 4 * e) * 4)) : *(const f32x4*)(x + c * 8 + 4 * e);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (c0 + u * TPB >= nch) continue;
      const float xe[8] = {xv[u][0].x, xv[u][0].y, xv[u][0].z, xv[u][0].w,
                           xv[u][1].x, xv[u][1].y, xv[u][1].z, xv[u][1].w};
#pragma unroll
      for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[r] = fmaf(__uint_as_float(wv[u][r][q] << 16), xe[2 * q], acc[r]);
          acc[r] = fmaf(__uint_as_float(wv[u][r][q] & 0xffff0000u), xe[2 * q + 1], acc[r]);
        }
    }
  }
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    float v = acc[r];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((tid & 63) == 0) red[tid >> 6][r] = v;
  }
  __syncthreads();
  if (tid < RW && row0 + tid < rows) {
    float v = 0.f;
    for (int w = 0; w < TPB / 64; ++w) v += red[w][tid];
    if (ydev)
      __hip_atomic_store(y + row0 + tid, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      y[row0 + tid] = v;
  }
}

__global__ __launch_bounds__(TPB) void k_stage1(const uint16_t* W, int K, const float* x, int rows, float* y) {
  gemv_rows<8, false>(W, K, x, blockIdx.x * 8, rows, y, false, nullptr);
}
__global__ __launch_bounds__(TPB) void k_stage2(const uint16_t* W, int K, const float* x, int rows, float* y) {
  gemv_rows<7, false>(W, K, x, blockIdx.x * 7, rows, y, false, nullptr);
}

// One launch: n1 first-stage workgroups, then the second stage's.  cnt: NCNT group counters
// (64 bytes apart) and a top counter; targets grow with the launch's epoch.  ACQ: after the
// wait, one agent-scope acquire and cached loads of y1 (else device-scope loads).
template <bool ACQ>
__global__ __launch_bounds__(TPB) void k_both(const uint16_t* W1, int K1, const float* x, int rows1, float* y1,
                                              const uint16_t* W2, int K2, int rows2, float* y2, unsigned* cnt,
                                              unsigned* fail, int n1, unsigned epoch) {
  const int b = blockIdx.x, tid = threadIdx.x;
  unsigned* top = cnt + 16 * NCNT;
  if (b < n1) {
    gemv_rows<8, false>(W1, K1, x, b * 8, rows1, y1, true, nullptr);
    if (tid == 0) {
      wait_mem();
      const int gi = b % NCNT;
      const unsigned per = (unsigned)(n1 / NCNT + (gi < n1 % NCNT ? 1 : 0));
      const unsigned t = __hip_atomic_fetch_add(cnt + 16 * gi, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (t == per * epoch - 1) __hip_atomic_fetch_add(top, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  const int row0 = (b - n1) * 7;
  u32x4 wpre[U][7];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int r = 0; r < 7; ++r)
      wpre[u][r] = ldnt(W2 + (size_t)min(row0 + r, rows2 - 1) * K2 + min(tid + u * TPB, K2 / 8 - 1) * 8);
  __shared__ int s_ok;
  if (tid == 0) {
    unsigned spins = 0;
    int ok = 1;
    while (__hip_atomic_load(top, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < (unsigned)NCNT * epoch) {
      __builtin_amdgcn_s_sleep(1);
      if (++spins > kSpinCap) {
        ok = 0;
        break;
      }
    }
    if (!ok) atomicOr(fail, 1u);
    s_ok = ok;
  }
  __syncthreads();
  if (!s_ok) return;
  if (ACQ) {
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    gemv_rows<7, false>(W2, K2, y1, row0, rows2, y2, false, wpre);
  } else {
    gemv_rows<7, true>(W2, K2, y1, row0, rows2, y2, false, wpre);
  }
}

static void dependent_products() {
  printf("## 5. two dependent weight-streaming products (7B gate/up- and down-shaped, batch 1)\n");
  const int R1 = 18944, K1 = 7168, R2 = 3584, K2 = 18944;
  uint16_t *W1, *W2;
  float *x, *y1, *y1f, *y2, *y2f;
  unsigned *cnt, *fail;
  CK(hipMalloc(&W1, (size_t)R1 * K1 * 2));
  CK(hipMalloc(&W2, (size_t)R2 * K2 * 2));
  CK(hipMalloc(&x, K1 * 4));
  CK(hipMalloc(&y1, R1 * 4));
  CK(hipMalloc(&y1f, R1 * 4));
  CK(hipMalloc(&y2, R2 * 4));
  CK(hipMalloc(&y2f, R2 * 4));
  CK(hipMalloc(&cnt, 16 * (NCNT + 1) * 4));
  CK(hipMalloc(&fail, 4));
  {
    std::vector<uint16_t> h((size_t)R1 * K1);
    unsigned s = 1;
    for (auto& v : h) {  // bf16 values of magnitude 1-2, random signs
      s = s * 1664525u + 1013904223u;
      v = (uint16_t)((0x3f80 + ((s >> 16) & 0x7f)) | ((s >> 31) << 15));
    }
    CK(hipMemcpy(W1, h.data(), h.size() * 2, hipMemcpyHostToDevice));
    CK(hipMemcpy(W2, h.data(), (size_t)R2 * K2 * 2, hipMemcpyHostToDevice));
    std::vector<float> hx(K1);
    for (auto& v : hx) {
      s = s * 1664525u + 1013904223u;
      v = ((s >> 8) & 0xffff) / 65536.f - 0.5f;
    }
    CK(hipMemcpy(x, hx.data(), K1 * 4, hipMemcpyHostToDevice));
  }
  CK(hipMemset(cnt, 0, 16 * (NCNT + 1) * 4));
  CK(hipMemset(fail, 0, 4));
  const int n1 = R1 / 8, n2 = (R2 + 6) / 7, reps = 50;
  hipEvent_t a, b;
  CK(hipEventCreate(&a));
  CK(hipEventCreate(&b));
  for (int i = 0; i < 5; ++i) {
    k_stage1<<<n1, TPB>>>(W1, K1, x, R1, y1);
    k_stage2<<<n2, TPB>>>(W2, K2, y1, R2, y2);
  }
  CK(hipDeviceSynchronize());
  CK(hipEventRecord(a));
  for (int i = 0; i < reps; ++i) k_stage1<<<n1, TPB>>>(W1, K1, x, R1, y1);
  CK(hipEventRecord(b));
  CK(hipDeviceSynchronize());
  printf("first product alone (271.6 MB):  %6.2f us\n", time_ms(a, b) * 1e3 / reps);
  CK(hipEventRecord(a));
  for (int i = 0; i < reps; ++i) k_stage2<<<n2, TPB>>>(W2, K2, y1, R2, y2);
  CK(hipEventRecord(b));
  CK(hipDeviceSynchronize());
  printf("second product alone (135.8 MB): %6.2f us\n", time_ms(a, b) * 1e3 / reps);
  CK(hipEventRecord(a));
  for (int i = 0; i < reps; ++i) {
    k_stage1<<<n1, TPB>>>(W1, K1, x, R1, y1);
    k_stage2<<<n2, TPB>>>(W2, K2, y1, R2, y2);
  }
  CK(hipEventRecord(b));
  CK(hipDeviceSynchronize());
  printf("two kernels:                     %6.2f us per pair\n", time_ms(a, b) * 1e3 / reps);
  std::vector<float> r2(R2), r2f(R2);
  CK(hipMemcpy(r2.data(), y2, R2 * 4, hipMemcpyDeviceToHost));
  unsigned epoch = 0;
  for (int acq = 0; acq < 2; ++acq) {
    auto kern = acq ? k_both<true> : k_both<false>;
    CK(hipMemset(y2f, 0, R2 * 4));
    for (int i = 0; i < 5; ++i) kern<<<n1 + n2, TPB>>>(W1, K1, x, R1, y1f, W2, K2, R2, y2f, cnt, fail, n1, ++epoch);
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(a));
    for (int i = 0; i < reps; ++i) kern<<<n1 + n2, TPB>>>(W1, K1, x, R1, y1f, W2, K2, R2, y2f, cnt, fail, n1, ++epoch);
    CK(hipEventRecord(b));
    CK(hipDeviceSynchronize());
    unsigned f = 0;
    CK(hipMemcpy(&f, fail, 4, hipMemcpyDeviceToHost));
    CK(hipMemcpy(r2f.data(), y2f, R2 * 4, hipMemcpyDeviceToHost));
    int diff = 0;
    for (int i = 0; i < R2; ++i) diff += r2[i] != r2f[i];
    printf("one launch, %-24s %6.2f us per pair; gave up %u; outputs unlike the two kernels' %d of %d\n",
           acq ? "acquire + cached loads:" : "device-scope loads:", time_ms(a, b) * 1e3 / reps, f, diff, R2);
  }
  printf("\n");
}

// ---------------------------------------------------------------- 6. memory-side cache
__global__ __launch_bounds__(TPB) void k_read_plain(const u32x4* p, size_t n16, unsigned* sink) {
  unsigned acc = 0;
  for (size_t i = (size_t)blockIdx.x * TPB + threadIdx.x; i < n16; i += (size_t)gridDim.x * TPB) {
    const u32x4 v = p[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == 0x9e3779b9u) sink[0] = acc;
}

static void cache_reuse() {
  printf("## 6. memory-side cache: one non-temporal read of a region, timed alone (event pair)\n");
  printf("(cold: after a 1 GiB read of other data; warm: right after a plain or non-temporal read\n"
         " of the same region; medians of 5 regions)\n");
  const size_t pool = (size_t)4 << 30, flush_bytes = (size_t)1 << 30;
  u32x4* p;
  unsigned* sink;
  CK(hipMalloc(&p, pool));
  CK(hipMalloc(&sink, 64));
  CK(hipMemset(p, 1, pool));
  CK(hipDeviceSynchronize());
  hipEvent_t a, b;
  CK(hipEventCreate(&a));
  CK(hipEventCreate(&b));
  const u32x4* flush = p + (pool - flush_bytes) / 16;  // the last GiB; the regions lie below 2 GiB
  auto flushc = [&]() {
    k_stream<<<2048, TPB>>>(flush, flush_bytes / 16, sink);
    CK(hipDeviceSynchronize());
  };
  auto timed = [&](const u32x4* q, size_t n16) {
    CK(hipEventRecord(a));
    k_stream<<<2048, TPB>>>(q, n16, sink);
    CK(hipEventRecord(b));
    CK(hipEventSynchronize(b));
    return (double)time_ms(a, b) * 1e3;
  };
  auto med = [](std::vector<double> v) {
    std::sort(v.begin(), v.end());
    return v[v.size() / 2];
  };
  printf("  size |  cold            | after plain read | after nt read\n");
  for (size_t mb : {8, 16, 32, 64, 128, 192}) {
    const size_t bytes = mb << 20, n16 = bytes / 16;
    std::vector<double> c, wp, wn;
    for (int rep = 0; rep < 5; ++rep) {
      const u32x4* r = p + (size_t)rep * ((size_t)256 << 20) / 16;
      flushc();
      c.push_back(timed(r, n16));
      flushc();
      k_read_plain<<<2048, TPB>>>(r, n16, sink);
      CK(hipDeviceSynchronize());
      wp.push_back(timed(r, n16));
      flushc();
      k_stream<<<2048, TPB>>>(r, n16, sink);
      CK(hipDeviceSynchronize());
      wn.push_back(timed(r, n16));
    }
    printf("%4zu MiB | %7.2f us %5.0f GB/s | %7.2f us %5.0f GB/s | %7.2f us %5.0f GB/s\n", mb, med(c), bytes / med(c) / 1e3,
           med(wp), bytes / med(wp) / 1e3, med(wn), bytes / med(wn) / 1e3);
  }
  printf("\n");
  CK(hipFree(p));
  CK(hipFree(sink));
}

int main() {
  hipDeviceProp_t prop;
  CK(hipGetDeviceProperties(&prop, 0));
  printf("# design probes on %s, %d compute units\n\n", prop.gcnArchName, prop.multiProcessorCount);
  stream_read();
  graph_boundary();
  {
    printf("## 3. cross-workgroup hand-off (each workgroup publishes 1 KB, the last reads them back)\n");
    float* data;
    unsigned *cnt, *err;
    CK(hipMalloc(&data, (size_t)1024 * TPB * 4));
    CK(hipMalloc(&cnt, 256));
    CK(hipMalloc(&err, 256));
    for (int N : {448, 768}) {
      publish<0>(N, data, cnt, err);
      publish<1>(N, data, cnt, err);
      publish<2>(N, data, cnt, err);
    }
    printf("\n## 4. grid barrier (cooperative launch, device-scope stores/loads, bounded spins)\n");
    float* slot;
    unsigned *bcnt, *fail;
    CK(hipMalloc(&slot, 4096 * 4));
    CK(hipMalloc(&bcnt, 64 * 4 * 80));
    CK(hipMalloc(&fail, 256));
    for (int N : {256, 512}) {
      barrier<false>(N, slot, bcnt, err, fail);
      barrier<true>(N, slot, bcnt, err, fail);
    }
    printf("\n");
  }
  dependent_products();
  cache_reuse();
  printf("done\n");
  return 0;
}
