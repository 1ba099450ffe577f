// Paged grouped-query attention over the KV cache (decode rows and probe chunks).
//
// Work: grid (workgroup split, kv head, row group).  A row group is the rows of one request
// in this forward (1 decode row, or the S rows of a probe chunk); its query columns are
// (row, query head of this kv head) pairs, padded to 16*NT.  Each of the 4 waves of a
// workgroup walks its own run of pages (split-K), so every K/V page is read once for all
// query columns of the request.  Per page (16 positions):
//   S^T[t][c] = K[t][:] . Q[c][:]   v_mfma_f32_16x16x32_bf16, A = K page, B = Q^T (bf16 hi+lo)
//   online softmax over t per column (exp2 domain), causal mask t <= pos(c)
//   O^T[d][c] += V^T[d][t] P^T[t][c] v_mfma_f32_16x16x16_bf16, B = P^T taken straight from
//                                    the S^T accumulator layout (bf16 hi+lo)
// The KV page layout makes every operand load a contiguous 1 KB (K) / 512 B (V) per wave
// instruction.  Waves merge (m, l, O) in LDS; when a (group, kv head) spans several
// workgroups their fp32 partials are combined by k_attn_merge, launched next.
#include <type_traits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace laser {

// Calls f(integral_constant<int, i>) for i = 0 .. N-1 (compile-time ring-buffer indices, so
// register arrays are never indexed dynamically).
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

__device__ __forceinline__ float safe_exp2(float x) { return x == -INFINITY ? 0.f : exp2f(x); }

template <class KT, int HD, int NT>
__global__ __launch_bounds__(64 * kAttnWaves) void k_attn(AttnArgs a) {
  constexpr int NS = HD / 32;  // QK k-steps
  constexpr int ND = HD / 16;  // PV d-tiles
  constexpr int NC = 16 * NT;  // padded query columns
  // Q (bf16 hi/lo) is only read in the page loop; the merge slots reuse the same LDS.
  constexpr int QBYTES = NC * HD * 2 * 2;
  constexpr int OBYTES = 2 * NC * HD * 4;
  __shared__ __align__(16) char s_raw[QBYTES > OBYTES ? QBYTES : OBYTES];
  uint16_t* s_qh = (uint16_t*)s_raw;
  uint16_t* s_ql = s_qh + NC * HD;
  float* const s_of = (float*)s_raw;  // merge slot k at s_of + k * NC * HD
  __shared__ int s_pos[NC];
  __shared__ float s_m[2][NC];
  __shared__ float s_l[2][NC];

  const GroupDesc gd = a.plan->groups[blockIdx.z];
  const int wg = blockIdx.x;
  if (wg >= gd.nwg) return;
  const int kvh = blockIdx.y;
  const int tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63;
  const int lc = l & 15, lg = l >> 4;
  const int NQ = gd.nrows * a.G;

  float m_run[NT], l_run[NT];
  f32x4 o[NT][ND];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    m_run[nt] = -INFINITY;
    l_run[nt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) o[nt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int split = wg * kAttnWaves + w;
  const int p0 = split * gd.pps;
  const int p1 = min(p0 + gd.pps, gd.npages);
  const int* btrow = a.bt + (size_t)gd.seq * a.max_pps;
  const size_t layer_base = (size_t)a.layer * a.num_pages;
  const size_t blk_elems = (size_t)16 * HD;

  // Page operands are loaded D pages ahead of their use into a ring of raw buffers (bf16
  // bits; fp32 pools are split into bf16 hi/lo when used).  With one query tile a wave's
  // whole run of pages is usually in flight at once.
  constexpr int D = (sizeof(KT) == 2 && NT == 1) ? 4 : 2;
  constexpr int KW = sizeof(KT) == 2 ? 1 : 2;  // 16-byte K loads per k-step
  u32x4 kraw[D][NS][KW];
  u32x4 vraw[D][ND];  // bf16: only the low 8 bytes are used
  auto load_page = [&](int pg, auto bufc) {
    constexpr int buf = decltype(bufc)::value;
    const int pid = btrow[pg];
    const size_t blk = ((layer_base + pid) * a.hkv + kvh) * blk_elems;
    if (sizeof(KT) == 2) {
      const uint16_t* kb = (const uint16_t*)a.kpool + blk;
      const uint16_t* vb = (const uint16_t*)a.vpool + blk;
#pragma unroll
      for (int s = 0; s < NS; ++s) kraw[buf][s][0] = ld_nt16(kb + s * 512 + 8 * l);
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const u32x2 t = ld_nt8(vb + dt * 256 + 4 * l);
        vraw[buf][dt] = u32x4{t[0], t[1], 0u, 0u};
      }
    } else {
      const float* kb = (const float*)a.kpool + blk;
      const float* vb = (const float*)a.vpool + blk;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        kraw[buf][s][0] = ld_nt16(kb + s * 512 + 8 * l);
        kraw[buf][s][KW - 1] = ld_nt16(kb + s * 512 + 8 * l + 4);
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) vraw[buf][dt] = ld_nt16(vb + dt * 256 + 4 * l);
    }
  };
  auto process_page = [&](int pg, auto cbc) {
    constexpr int cb = decltype(cbc)::value;
    // K operand: lane l holds K[t = l%16][d = 32s + 8(l/16) + j]; V^T: V[t = 4(l/16) + j][16dt + l%16]
    bf16x8 khi[NS], klo[NS];
    s16x4 vhi[ND], vlo[ND];
    if (sizeof(KT) == 2) {
#pragma unroll
      for (int s = 0; s < NS; ++s) khi[s] = __builtin_bit_cast(bf16x8, kraw[cb][s][0]);
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) vhi[dt] = __builtin_bit_cast(s16x4, u32x2{vraw[cb][dt][0], vraw[cb][dt][1]});
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const u32x4 x0 = kraw[cb][s][0], x1 = kraw[cb][s][KW - 1];
        u32x4 ph, pl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint16_t h0, l0, h1, l1;
          const u32x4& src = q < 2 ? x0 : x1;
          split_bf16(__uint_as_float(src[(q & 1) * 2]), h0, l0);
          split_bf16(__uint_as_float(src[(q & 1) * 2 + 1]), h1, l1);
          ph[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
          pl[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        }
        khi[s] = __builtin_bit_cast(bf16x8, ph);
        klo[s] = __builtin_bit_cast(bf16x8, pl);
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const u32x4 x = vraw[cb][dt];
        s16x4 h4, l4;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint16_t hh, ll;
          split_bf16(__uint_as_float(x[q]), hh, ll);
          h4[q] = (short)hh;
          l4[q] = (short)ll;
        }
        vhi[dt] = h4;
        vlo[dt] = l4;
      }
    }
    // Slots past the group's last position hold no written value (possibly not even a
    // finite one); P is zero there but 0 * NaN is not, so those V entries are zeroed.
    if (pg * 16 + 15 > gd.maxpos) {
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (pg * 16 + 4 * lg + j > gd.maxpos) {
            vhi[dt][j] = 0;
            if (sizeof(KT) == 4) vlo[dt][j] = 0;
          }
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (nt * 16 >= NQ) break;
      f32x4 sacc = f32x4{0.f, 0.f, 0.f, 0.f};
      const int qrow = (nt * 16 + lc) * HD;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8 qh = *(const bf16x8*)(s_qh + qrow + 32 * s + 8 * lg);
        const bf16x8 ql = *(const bf16x8*)(s_ql + qrow + 32 * s + 8 * lg);
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(khi[s], qh, sacc, 0, 0, 0);
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(khi[s], ql, sacc, 0, 0, 0);
        if (sizeof(KT) == 4) sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(klo[s], qh, sacc, 0, 0, 0);
      }
      // lane (c = lc, lg): sacc[i] = score of position pg*16 + 4*lg + i for column c
      const int cpos = s_pos[nt * 16 + lc];
      float sv[4];
      float mloc = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tg = pg * 16 + 4 * lg + i;
        sv[i] = (tg <= cpos) ? sacc[i] * a.scale_log2 : -INFINITY;
        mloc = fmaxf(mloc, sv[i]);
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
      const float m_new = fmaxf(m_run[nt], mloc);
      const float alpha = (m_new == -INFINITY) ? 1.f : safe_exp2(m_run[nt] - m_new);
      float pv[4], ls = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pv[i] = (sv[i] == -INFINITY) ? 0.f : exp2f(sv[i] - m_new);
        ls += pv[i];
      }
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      l_run[nt] = l_run[nt] * alpha + ls;
      m_run[nt] = m_new;
      s16x4 phi, plo;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint16_t hh, ll;
        split_bf16(pv[i], hh, ll);
        phi[i] = (short)hh;
        plo[i] = (short)ll;
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        o[nt][dt] *= alpha;
        o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vhi[dt], phi, o[nt][dt], 0, 0, 0);
        o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vhi[dt], plo, o[nt][dt], 0, 0, 0);
        if (sizeof(KT) == 4) o[nt][dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vlo[dt], phi, o[nt][dt], 0, 0, 0);
      }
    }
  };
  static_for<D>([&](auto b) {
    if (p0 + (int)b < p1) load_page(p0 + (int)b, b);
  });
  // queries are staged while the first pages are in flight
  for (int idx = tid; idx < NC * HD; idx += blockDim.x) {
    const int c = idx / HD, d = idx - c * HD;
    float v = 0.f;
    if (c < NQ) {
      const int row = gd.row0 + c / a.G;
      const int head = kvh * a.G + c % a.G;
      v = a.q[((size_t)row * a.hq + head) * HD + d];
    }
    uint16_t hi, lo;
    split_bf16(v, hi, lo);
    s_qh[idx] = hi;
    s_ql[idx] = lo;
  }
  for (int c = tid; c < NC; c += blockDim.x) s_pos[c] = c < NQ ? a.plan->rows[gd.row0 + c / a.G].pos : -1;
  __syncthreads();

  for (int base = p0; base < p1; base += D) {
    static_for<D>([&](auto b) {
      const int pg = base + (int)b;
      if (pg < p1) {
        process_page(pg, b);
        if (pg + D < p1) load_page(pg + D, b);
      }
    });
  }

  // ---- merge the 4 waves in two rounds through 2 LDS slots
  auto publish = [&](int slot) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int c = nt * 16 + lc;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) s_of[slot * NC * HD + c * HD + 16 * dt + 4 * lg + i] = o[nt][dt][i];
      if (lg == 0) {
        s_m[slot][c] = m_run[nt];
        s_l[slot][c] = l_run[nt];
      }
    }
  };
  auto absorb = [&](int slot) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int c = nt * 16 + lc;
      const float m2 = s_m[slot][c], l2 = s_l[slot][c];
      const float mm = fmaxf(m_run[nt], m2);
      const float ca = (mm == -INFINITY) ? 0.f : safe_exp2(m_run[nt] - mm);
      const float cb = (mm == -INFINITY) ? 0.f : safe_exp2(m2 - mm);
      l_run[nt] = l_run[nt] * ca + l2 * cb;
      m_run[nt] = mm;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) o[nt][dt][i] = o[nt][dt][i] * ca + s_of[slot * NC * HD + c * HD + 16 * dt + 4 * lg + i] * cb;
    }
  };
  __syncthreads();  // every wave is done with Q before the slots overwrite it
  if (w >= 2) publish(w - 2);
  __syncthreads();
  if (w < 2) absorb(w);
  __syncthreads();
  if (w == 1) publish(0);
  __syncthreads();
  if (w == 0) {
    absorb(0);
    publish(1);  // workgroup result (unnormalised) in slot 1
  }
  __syncthreads();

  const int ncols = a.max_rows * a.G;
  if (gd.nwg == 1) {
    for (int idx = tid; idx < NQ * HD; idx += blockDim.x) {
      const int c = idx / HD, d = idx - c * HD;
      const int row = gd.row0 + c / a.G, head = kvh * a.G + c % a.G;
      a.o[((size_t)row * a.hq + head) * HD + d] = s_of[1 * NC * HD + c * HD + d] / s_l[1][c];
    }
    return;
  }
  const size_t slot_base = ((size_t)kvh * kAttnMaxWG + wg) * ncols + (size_t)gd.row0 * a.G;
  for (int idx = tid; idx < NQ * HD; idx += blockDim.x) a.part[slot_base * HD + idx] = s_of[1 * NC * HD + idx];
  for (int c = tid; c < NQ; c += blockDim.x) {
    a.ml[(slot_base + c) * 2 + 0] = s_m[1][c];
    a.ml[(slot_base + c) * 2 + 1] = s_l[1][c];
  }
}

// Combines the workgroup partials (m, l, O) of every (row, query head) whose group used
// more than one attention workgroup: o = sum_w O_w 2^(m_w - M) / sum_w l_w 2^(m_w - M),
// M = max_w m_w.  grid (rows, query heads), 16 waves: wave v takes partials w = v mod 16
// (all loads of a wave issued together, before the plan lookup), lanes take dims; the
// waves are then combined in LDS in fixed order.
constexpr int kMergeWaves = 16;
__global__ __launch_bounds__(64 * kMergeWaves) void k_attn_merge(AttnArgs a, int hd) {
  constexpr int PER = kAttnMaxWG / kMergeWaves;
  __shared__ float s_m[kMergeWaves], s_l[kMergeWaves];
  __shared__ float s_o[kMergeWaves][128];
  const int row = blockIdx.x, head = blockIdx.y;
  const int v = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int kvh = head / a.G, gi = head - kvh * a.G;
  const size_t ncols = (size_t)a.max_rows * a.G;
  const size_t col = (size_t)row * a.G + gi;
  // every slot is loaded before the group's workgroup count is known (slots past it are
  // replaced below, never combined), so the loads overlap the plan lookup
  float mv[PER], lv[PER], o0[PER], o1[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const size_t sb = ((size_t)kvh * kAttnMaxWG + v + kMergeWaves * i) * ncols + col;
    mv[i] = a.ml[sb * 2];
    lv[i] = a.ml[sb * 2 + 1];
    o0[i] = a.part[sb * hd + l];
    o1[i] = (l + 64 < hd) ? a.part[sb * hd + l + 64] : 0.f;
  }
  const Plan* plan = a.plan;
  int z = 0;
  while (z + 1 < plan->n_groups && plan->groups[z + 1].row0 <= row) ++z;
  const int nwg = plan->groups[z].nwg;
  if (nwg <= 1) return;  // written directly by the attention kernel
#pragma unroll
  for (int i = 0; i < PER; ++i)
    if (v + kMergeWaves * i >= nwg) {
      mv[i] = -INFINITY;
      lv[i] = 0.f;
      o0[i] = o1[i] = 0.f;
    }
  float M = -INFINITY;
#pragma unroll
  for (int i = 0; i < PER; ++i) M = fmaxf(M, mv[i]);
  float L = 0.f, O0 = 0.f, O1 = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const float f = (M == -INFINITY) ? 0.f : safe_exp2(mv[i] - M);
    L += lv[i] * f;
    O0 += o0[i] * f;
    O1 += o1[i] * f;
  }
  if (l == 0) {
    s_m[v] = M;
    s_l[v] = L;
  }
  s_o[v][l] = O0;
  s_o[v][l + 64] = O1;
  __syncthreads();
  if (v == 0) {
    float Mt = -INFINITY;
#pragma unroll
    for (int u = 0; u < kMergeWaves; ++u) Mt = fmaxf(Mt, s_m[u]);
    float Lt = 0.f, Ot0 = 0.f, Ot1 = 0.f;
#pragma unroll
    for (int u = 0; u < kMergeWaves; ++u) {
      const float f = (s_m[u] == -INFINITY) ? 0.f : safe_exp2(s_m[u] - Mt);
      Lt += s_l[u] * f;
      Ot0 += s_o[u][l] * f;
      Ot1 += s_o[u][l + 64] * f;
    }
    float* out = a.o + ((size_t)row * a.hq + head) * hd;
    out[l] = Ot0 / Lt;
    if (l + 64 < hd) out[l + 64] = Ot1 / Lt;
  }
}

hipError_t launch_attn_merge(const AttnArgs& a, int M, int hd, hipStream_t s) {
  return launch_k(k_attn_merge, dim3(M, a.hq), dim3(64 * kMergeWaves), s, a, hd);
}

template <class KT, int HD>
static hipError_t launch_nt(int nt, const AttnArgs& a, dim3 grid, hipStream_t s) {
  const dim3 block(64 * kAttnWaves);
  switch (nt) {
    case 1: return launch_k(k_attn<KT, HD, 1>, grid, block, s, a);
    case 2: return launch_k(k_attn<KT, HD, 2>, grid, block, s, a);
    case 4: return launch_k(k_attn<KT, HD, 4>, grid, block, s, a);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attn(int dtype, int hd, int nt, const AttnArgs& a, dim3 grid, hipStream_t s) {
  if (dtype == 1) {
    if (hd == 128) return launch_nt<bf16_t, 128>(nt, a, grid, s);
    if (hd == 64) return launch_nt<bf16_t, 64>(nt, a, grid, s);
  } else {
    if (hd == 128) return launch_nt<float, 128>(nt, a, grid, s);
    if (hd == 64) return launch_nt<float, 64>(nt, a, grid, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace laser
