// Paged grouped-query attention over the KV cache (decode rows and probe chunks).
//
// Work: grid (work item, kv head).  A row group is contiguous rows over one page range of one
// block table (the rows of a request in this forward, or of a request and its forks over
// their shared pages); its query columns are (row, query head of this kv head) pairs in
// 16-column tiles.  A work item is one tile of a group over one page split: each of the
// workgroup's 4 waves walks its own run of pages (split-K) and the waves merge (m, l, O) in
// one LDS round.  The host lists the tiles of one split 8 items apart: workgroups go to the
// 8 XCDs in turn, so these land on one XCD and each page comes from HBM once into that XCD's
// L2 for all of the group's columns.  Per page (16 positions):
//   S^T[t][c] = K[t][:] . Q[c][:]   v_mfma_f32_16x16x32_bf16, A = K page, B = Q^T (bf16 hi+lo)
//   online softmax over t per column (exp2 domain), causal mask t <= pos(c)
//   O^T[d][c] += V^T[d][t] P^T[t][c] v_mfma_f32_16x16x16_bf16, B = P^T taken straight from
//                                    the S^T accumulator layout (bf16 hi+lo)
// The KV page layout makes every operand load a contiguous 1 KB (K) / 512 B (V) per wave
// instruction.  A wave's query tile stays in registers and pages are taken in pairs, so the
// cross-lane max and sum reductions run once per 32 positions.  When a (group, kv head)
// spans several workgroups their fp32 partials are combined: for a one-row group (a decode
// row) by the group's last workgroup to finish, inside this kernel (the partials go out with
// device-scope stores, an arrival counter tells the last one; see the fused items below);
// otherwise by k_attn_merge, launched next.
#include <type_traits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace laser {

__device__ __forceinline__ float safe_exp2(float x) { return x == -INFINITY ? 0.f : exp2f(x); }

template <class KT, int HD>
__global__ __launch_bounds__(64 * kAttnWaves) void k_attn(AttnArgs a) {
  constexpr int NS = HD / 32;  // QK k-steps
  constexpr int ND = HD / 16;  // PV d-tiles
  constexpr int NC = 16;       // query columns of the tile
  // LDS: the tile's queries (bf16 hi/lo) and the merge slots of waves 1-3.  Rows are padded by 16 bytes, so the 16 columns a wave reads at
  // once (row stride) fall in 16 different bank groups instead of one.
  constexpr int QS = HD + 8;  // query row stride (bf16 elements)
  constexpr int OS = HD + 4;  // merge-slot row stride (floats)
  __shared__ __align__(16) uint16_t s_qh[NC * QS];
  __shared__ __align__(16) uint16_t s_ql[NC * QS];
  __shared__ __align__(16) float s_of[3 * 16 * OS];  // slot k at s_of + k * 16 * OS
  __shared__ int s_pos[NC];
  __shared__ float s_m[3][16];
  __shared__ float s_l[3][16];

  const AttnItem wi = a.plan->items[blockIdx.x];
  if (wi.nrows == 0) return;  // padding item
  const int nrows = wi.nrows & 0xff;
  const int fuse_n = (wi.nrows >> 8) & 0xff;  // fused group: its split count (else 0)
  const int NQ = nrows * a.G;
  const int kvh = blockIdx.y;
  const int tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63;
  const int lc = l & 15, lg = l >> 4;
  const int col0 = (wi.info & 0xff) * 16;  // the tile's first query column

  // Wave w walks its run of the item's pages for the tile's 16 columns, then the waves merge
  // through LDS.
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int p0 = wi.p0 + w * wi.pps;
  const int p1 = min(p0 + wi.pps, wi.pend);
  const int* btrow = a.bt + (size_t)wi.seq * a.max_pps;
  const size_t layer_base = (size_t)a.layer * a.num_pages;
  const size_t blk_elems = (size_t)16 * HD;

  // The page ids of this wave's run are read up front, together with the queries, so no
  // page load waits behind another page's data (vector-memory counters complete in order).
  // (Named values, not an array: an indexed array goes to scratch memory, whose accesses
  // share the in-order counter with the page loads.)
  const int plast = max(p1 - 1, 0);  // clamped, branch-free: the loads issue back to back
  const int pid0 = btrow[min(p0, plast)], pid1 = btrow[min(p0 + 1, plast)];
  const int pid2 = btrow[min(p0 + 2, plast)], pid3 = btrow[min(p0 + 3, plast)];
  auto page_id = [&](int pg) -> int {  // pg is wave-uniform
    const int k = pg - p0;
    return k == 0 ? pid0 : k == 1 ? pid1 : k == 2 ? pid2 : k == 3 ? pid3 : btrow[pg];
  };
  constexpr int Q4 = NC * HD / 4 / (64 * kAttnWaves);  // query float4 loads per thread
  static_assert(Q4 * 4 * 64 * kAttnWaves == NC * HD, "query tile");
  float4 qv[Q4];
#pragma unroll
  for (int i = 0; i < Q4; ++i) {  // padding columns load the last real one, zeroed when staged
    const int idx = 4 * (tid + i * 64 * kAttnWaves);
    const int c = min(col0 + idx / HD, NQ - 1), d = idx % HD;
    const int row = wi.row0 + c / a.G;
    const int head = kvh * a.G + c % a.G;
    qv[i] = *(const float4*)(a.q + ((size_t)row * a.hq + head) * HD + d);
  }
  static_assert(NC <= 64 * kAttnWaves, "one position per thread");
  const int cpos_loaded = a.plan->rows[wi.row0 + min(col0 + tid, NQ - 1) / a.G].pos;  // column tid's position

  // Page operands are loaded D pages ahead of their use into a ring of raw buffers (bf16
  // bits; fp32 pools are split into bf16 hi/lo when used).  A decode split is usually two
  // pages, so its whole run is in flight at once.
  constexpr int D = 2;
  constexpr int KW = sizeof(KT) == 4 ? 2 : 1;  // 16-byte K loads per k-step (fp8: one 8-byte load)
  // raw page words per lane, sized to what each storage type loads (registers are what
  // limits how many waves a CU holds)
  using KRaw = std::conditional_t<sizeof(KT) == 1, u32x2, u32x4>;
  using VRaw = std::conditional_t<sizeof(KT) == 1, uint32_t, std::conditional_t<sizeof(KT) == 2, u32x2, u32x4>>;
  KRaw kraw[D][NS][KW];
  VRaw vraw[D][ND];
  auto load_page = [&](int pg, auto bufc) {
    constexpr int buf = decltype(bufc)::value;
    const int pid = page_id(pg);
    const size_t blk = ((layer_base + pid) * a.hkv + kvh) * blk_elems;
    if constexpr (sizeof(KT) == 1) {
      const uint8_t* kb = (const uint8_t*)a.kpool + blk;
      const uint8_t* vb = (const uint8_t*)a.vpool + blk;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const u32x2 t = ld_nt8(kb + s * 512 + 8 * l);
        kraw[buf][s][0] = t;
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
        vraw[buf][dt] = __builtin_nontemporal_load((const uint32_t*)(vb + dt * 256 + 4 * l));
    } else if constexpr (sizeof(KT) == 2) {
      const uint16_t* kb = (const uint16_t*)a.kpool + blk;
      const uint16_t* vb = (const uint16_t*)a.vpool + blk;
#pragma unroll
      for (int s = 0; s < NS; ++s) kraw[buf][s][0] = ld_nt16(kb + s * 512 + 8 * l);
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const u32x2 t = ld_nt8(vb + dt * 256 + 4 * l);
        vraw[buf][dt] = t;
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
  // MFMA operands of one page.  K: lane l holds K[t = l%16][d = 32s + 8(l/16) + j];
  // V^T: V[t = 4(l/16) + j][d = 16dt + l%16].  Slots past the group's last position hold no
  // written value (possibly not even a finite one); P is zero there but 0 * NaN is not, so
  // those V entries are zeroed.
  struct PageOps {
    bf16x8 khi[NS], klo[NS];
    s16x4 vhi[ND], vlo[ND];
  };
  auto unpack = [&](int pg, auto cbc, PageOps& P) {
    constexpr int cb = decltype(cbc)::value;
    if constexpr (sizeof(KT) == 1) {  // E4M3 -> bf16 is exact: no lo part
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        uint32_t w0, w1, w2, w3;
        fp8x4_to_bf16x4(kraw[cb][s][0][0], w0, w1);
        fp8x4_to_bf16x4(kraw[cb][s][0][1], w2, w3);
        P.khi[s] = __builtin_bit_cast(bf16x8, u32x4{w0, w1, w2, w3});
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        uint32_t w0, w1;
        fp8x4_to_bf16x4(vraw[cb][dt], w0, w1);
        P.vhi[dt] = __builtin_bit_cast(s16x4, u32x2{w0, w1});
      }
    } else if constexpr (sizeof(KT) == 2) {
#pragma unroll
      for (int s = 0; s < NS; ++s) P.khi[s] = __builtin_bit_cast(bf16x8, kraw[cb][s][0]);
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) P.vhi[dt] = __builtin_bit_cast(s16x4, vraw[cb][dt]);
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
        P.khi[s] = __builtin_bit_cast(bf16x8, ph);
        P.klo[s] = __builtin_bit_cast(bf16x8, pl);
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
        P.vhi[dt] = h4;
        P.vlo[dt] = l4;
      }
    }
    if (pg * 16 + 15 > wi.maxpos) {
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (pg * 16 + 4 * lg + j > wi.maxpos) {
            P.vhi[dt][j] = 0;
            if (sizeof(KT) == 4) P.vlo[dt][j] = 0;
          }
    }
  };
  // S^T tile of one page: lane (c = lc, lg) gets the scores of positions 16pg + 4lg + i.
  // (The hi and lo query parts accumulate in two chains, summed at the end, so that
  // consecutive matrix-core ops do not wait for each other's results.)
  auto scores = [&](const PageOps& P, const bf16x8* qh, const bf16x8* ql) {
    f32x4 shi = f32x4{0.f, 0.f, 0.f, 0.f}, slo = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      shi = __builtin_amdgcn_mfma_f32_16x16x32_bf16(P.khi[s], qh[s], shi, 0, 0, 0);
      slo = __builtin_amdgcn_mfma_f32_16x16x32_bf16(P.khi[s], ql[s], slo, 0, 0, 0);
      if (sizeof(KT) == 4) slo = __builtin_amdgcn_mfma_f32_16x16x32_bf16(P.klo[s], qh[s], slo, 0, 0, 0);
    }
    return shi + slo;
  };
  // O^T += V^T P^T for one page; P^T comes straight from the score accumulator layout.
  auto accumulate = [&](const PageOps& P, const float* pv, f32x4* acc) {
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
      acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(P.vhi[dt], phi, acc[dt], 0, 0, 0);
      acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(P.vhi[dt], plo, acc[dt], 0, 0, 0);
      if (sizeof(KT) == 4) acc[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(P.vlo[dt], phi, acc[dt], 0, 0, 0);
    }
  };

  // The first D pages load unconditionally (a run shorter than D loads its last page again,
  // unused): a branch here would make the wait for page 1's id also wait for page 0's data.
  static_for<D>([&](auto b) { load_page(min(p0 + (int)b, plast), b); });
  // Queries (loaded above, with the page ids) are split into bf16 hi/lo in LDS while the
  // first pages are in flight.
  {
#pragma unroll
    for (int i = 0; i < Q4; ++i) {
      const int idx = 4 * (tid + i * 64 * kAttnWaves);
      const bool real = col0 + idx / HD < NQ;
      const float x[4] = {real ? qv[i].x : 0.f, real ? qv[i].y : 0.f, real ? qv[i].z : 0.f, real ? qv[i].w : 0.f};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint16_t hi, lo;
        split_bf16(x[e], hi, lo);
        s_qh[(idx / HD) * QS + idx % HD + e] = hi;
        s_ql[(idx / HD) * QS + idx % HD + e] = lo;
      }
    }
  }
  if (tid < NC) s_pos[tid] = col0 + tid < NQ ? cpos_loaded : -1;
  __syncthreads();

  // pages in pairs: one max and one sum reduction across the lane groups per 32 positions
  const int c = col0 + lc;  // this lane's query column
  bf16x8 qh[NS], ql[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    qh[s] = *(const bf16x8*)(s_qh + lc * QS + 32 * s + 8 * lg);
    ql[s] = *(const bf16x8*)(s_ql + lc * QS + 32 * s + 8 * lg);
  }
  const int cpos = s_pos[lc];
  auto pair = [&](int pgA, auto ca, auto cbB) {
    const int pgB = pgA + 1;
    const bool hasB = pgB < p1;  // wave-uniform
    PageOps A, B;
    unpack(pgA, ca, A);
    const f32x4 sa = scores(A, qh, ql);
    f32x4 sb = f32x4{0.f, 0.f, 0.f, 0.f};
    if (hasB) {
      unpack(pgB, cbB, B);
      sb = scores(B, qh, ql);
    }
    float sv[8];
    float mloc = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ta = pgA * 16 + 4 * lg + i, tb = pgB * 16 + 4 * lg + i;
      sv[i] = (ta <= cpos) ? sa[i] * a.scale_log2 : -INFINITY;
      sv[4 + i] = (hasB && tb <= cpos) ? sb[i] * a.scale_log2 : -INFINITY;
      mloc = fmaxf(mloc, fmaxf(sv[i], sv[4 + i]));
    }
    mloc = max_x16(mloc);
    mloc = max_x32(mloc);
    const float m_new = fmaxf(m_run, mloc);
    // o and l are still zero while m_run is -inf, so they need no rescale then
    const bool grow = m_run != -INFINITY && m_new != m_run;
    const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.f;
    float pv[8], ls = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      pv[i] = (sv[i] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(sv[i] - m_new);
      ls += pv[i];
    }
    ls = sum_x16(ls);
    ls = sum_x32(ls);
    l_run = l_run * alpha + ls;
    m_run = m_new;
    if (__builtin_amdgcn_read_exec() & __ballot(grow)) {  // any lane whose max moved
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) o[dt] *= alpha;
    }
    accumulate(A, pv, o);
    if (hasB) accumulate(B, pv + 4, o);
  };
  for (int base = p0; base < p1; base += D) {
    static_for<D / 2>([&](auto h) {
      constexpr int bA = 2 * decltype(h)::value;
      const int pg = base + bA;
      if (pg < p1) {
        pair(pg, std::integral_constant<int, bA>{}, std::integral_constant<int, bA + 1>{});
        if (pg + D < p1) load_page(pg + D, std::integral_constant<int, bA>{});
        if (pg + 1 + D < p1) load_page(pg + 1 + D, std::integral_constant<int, bA + 1>{});
      }
    });
  }

  // ---- one-round merge of the page-parallel waves: 1-3 publish, 0 absorbs in order
  if (w > 0) {
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) *(f32x4*)(s_of + (w - 1) * 16 * OS + lc * OS + 16 * dt + 4 * lg) = o[dt];
    if (lg == 0) {
      s_m[w - 1][lc] = m_run;
      s_l[w - 1][lc] = l_run;
    }
  }
  __syncthreads();
  if (w != 0 && fuse_n == 0) return;
  const size_t ncols = (size_t)a.max_rows * a.G;
  const __amdgpu_buffer_rsrc_t rpart = dev_rsrc(a.part, a.part_bytes), rml = dev_rsrc(a.ml, a.ml_bytes);
  if (w == 0) {
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      const float m2 = s_m[u][lc], l2 = s_l[u][lc];
      const float mm = fmaxf(m_run, m2);
      const float ca = (mm == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - mm);
      const float cb2 = (mm == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m2 - mm);
      l_run = l_run * ca + l2 * cb2;
      m_run = mm;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const f32x4 x = *(const f32x4*)(s_of + u * 16 * OS + lc * OS + 16 * dt + 4 * lg);
        o[dt] = o[dt] * ca + x * cb2;
      }
    }
    // ---- the tile's columns: the output (one workgroup) or the workgroup's partial
    if (c < NQ) {
      const int row = wi.row0 + c / a.G, head = kvh * a.G + c % a.G;
      const size_t col = ((size_t)kvh * kAttnMaxWG + ((wi.info >> 8) & 0xffff)) * ncols + (size_t)wi.row0 * a.G + c;
      if (wi.info & (1 << 24)) {
        float* out = a.o + ((size_t)row * a.hq + head) * HD;
        const float inv = 1.f / l_run;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) *(f32x4*)(out + 16 * dt + 4 * lg) = o[dt] * inv;
      } else if (fuse_n) {  // device-scope stores: another XCD's workgroup may merge them
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) st_dev16(rpart, (uint32_t)((col * HD + 16 * dt + 4 * lg) * 4), o[dt]);
        if (lg == 0) st_dev8(rml, (uint32_t)(col * 8), m_run, l_run);
      } else {
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) *(f32x4*)(a.part + col * HD + 16 * dt + 4 * lg) = o[dt];
        if (lg == 0) {
          a.ml[col * 2 + 0] = m_run;
          a.ml[col * 2 + 1] = l_run;
        }
      }
    }
  }
  if (fuse_n == 0) return;

  // ---- fused group: count this workgroup's arrival once its partial is stored; the last of
  // the group's fuse_n workgroups combines every split (slots 0 .. fuse_n-1, fixed order):
  // o = sum_s O_s 2^(m_s - M) / sum_s l_s 2^(m_s - M), then re-arms the counter.
  __shared__ unsigned s_tk;
  unsigned* cnt = a.cnt + ((size_t)kvh * kMaxGroups + (wi.nrows >> 16)) * kAttnCntStride;
  if (w == 0) {
    wait_mem();
    if (l == 0) s_tk = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (s_tk != (unsigned)(fuse_n - 1)) return;
  constexpr int CH = HD / 4;  // 4-dim chunks of a column
  if (tid < NQ * CH) {
    const int cc = tid / CH, d4 = tid - cc * CH;
    const size_t colb = (size_t)wi.row0 * a.G + cc;
    float M = -INFINITY, Ls = 0.f;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    constexpr int B = 8;  // slots loaded together
    for (int s0 = 0; s0 < fuse_n; s0 += B) {
      f32x4 ov[B];
      i32x2 mv[B];
#pragma unroll
      for (int j = 0; j < B; ++j) {  // past the count: slot fuse_n - 1 again (ignored below)
        const size_t colx = ((size_t)kvh * kAttnMaxWG + min(s0 + j, fuse_n - 1)) * ncols + colb;
        ov[j] = ld_dev16(rpart, (uint32_t)((colx * HD + 4 * d4) * 4));
        mv[j] = ld_dev8(rml, (uint32_t)(colx * 8));
      }
#pragma unroll
      for (int j = 0; j < B; ++j) {
        if (s0 + j < fuse_n) {
          const float ms = __int_as_float(mv[j][0]), ls = __int_as_float(mv[j][1]);
          const float mn = fmaxf(M, ms);
          const float ca = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - mn);
          const float cb = (ms == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ms - mn);
          Ls = Ls * ca + ls * cb;
          acc = acc * ca + ov[j] * cb;
          M = mn;
        }
      }
    }
    const int row = wi.row0 + cc / a.G, head = kvh * a.G + cc % a.G;
    *(f32x4*)(a.o + ((size_t)row * a.hq + head) * HD + 4 * d4) = acc * (1.f / Ls);
  }
  if (tid == 0) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Combines the workgroup partials (m, l, O) of every (row, query head) whose group used
// more than one attention workgroup: o = sum_w O_w 2^(m_w - M) / sum_w l_w 2^(m_w - M),
// M = max_w m_w.  grid (rows, query heads), 8 waves.  A slot's HD floats are read by HD/4
// consecutive lanes with 16-byte loads, each lane also reading the slot's (m, l) pair, so
// one wave load covers 64/(HD/4) slots; a lane takes kAttnMaxWG/(kMergeWaves x that) slots, all its
// loads issued together before the plan lookup.  Each wave combines its slots across its
// lanes, then the waves are combined in LDS in fixed order.
constexpr int kMergeWaves = 8;
template <int HD>
__global__ __launch_bounds__(64 * kMergeWaves) void k_attn_merge(AttnArgs a, int nslots) {
  constexpr int LPS = HD / 4;             // lanes per slot
  constexpr int SPW = 64 / LPS;           // slots per wave load
  constexpr int SPP = SPW * kMergeWaves;  // slots per workgroup pass
  constexpr int PER = kAttnMaxWG / SPP;   // slots per lane
  static_assert(PER * SPP == kAttnMaxWG, "slot passes");
  __shared__ float s_m[kMergeWaves], s_l[kMergeWaves];
  __shared__ __align__(16) float s_o[kMergeWaves][HD];
  const int row = blockIdx.x, head = blockIdx.y;
  const int v = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int d4 = l % LPS, sl = l / LPS;
  const int kvh = head / a.G, gi = head - kvh * a.G;
  const size_t ncols = (size_t)a.max_rows * a.G;
  const size_t col = (size_t)row * a.G + gi;
  // Slots at or past nslots (the launch's bound on every group's count) read slot
  // nslots - 1 again, a cached line, instead of stale partials; slots past the row's own
  // count are replaced below, never combined.  The loads stay unconditional so none waits
  // for another.
  float mv[PER], lv[PER];
  f32x4 ov[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int slot = min(SPP * i + SPW * v + sl, nslots - 1);
    const size_t sb = ((size_t)kvh * kAttnMaxWG + slot) * ncols + col;
    const float2 ml = *(const float2*)(a.ml + sb * 2);
    mv[i] = ml.x;
    lv[i] = ml.y;
    ov[i] = *(const f32x4*)(a.part + sb * HD + 4 * d4);
  }
  const int nwg = a.plan->row_nslots[row];
  if (nwg <= 1) return;  // written directly by the attention kernel
#pragma unroll
  for (int i = 0; i < PER; ++i)
    if (SPP * i + SPW * v + sl >= nwg) {
      mv[i] = -INFINITY;
      lv[i] = 0.f;
      ov[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  float M = -INFINITY;
#pragma unroll
  for (int i = 0; i < PER; ++i) M = fmaxf(M, mv[i]);
  M = wave_max(M);  // over the wave's slots
  float L = 0.f;
  f32x4 O = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const float f = (M == -INFINITY) ? 0.f : safe_exp2(mv[i] - M);
    L += lv[i] * f;
    O += ov[i] * f;
  }
  // the wave's slot lanes (LPS apart) summed, so every lane holds the wave's totals
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
  const int d = threadIdx.x;
  if (d < HD) {
    float Mt = -INFINITY;
#pragma unroll
    for (int u = 0; u < kMergeWaves; ++u) Mt = fmaxf(Mt, s_m[u]);
    float Lt = 0.f, Ot = 0.f;
#pragma unroll
    for (int u = 0; u < kMergeWaves; ++u) {
      const float f = (s_m[u] == -INFINITY) ? 0.f : safe_exp2(s_m[u] - Mt);
      Lt += s_l[u] * f;
      Ot += s_o[u][d] * f;
    }
    a.o[((size_t)row * a.hq + head) * HD + d] = Ot / Lt;
  }
}

hipError_t launch_attn_merge(const AttnArgs& a, int M, int hd, int nslots, hipStream_t s) {
  if (nslots < 1 || nslots > kAttnMaxWG) return hipErrorInvalidValue;
  if (hd == 128) return launch_k(k_attn_merge<128>, dim3(M, a.hq), dim3(64 * kMergeWaves), s, a, nslots);
  if (hd == 64) return launch_k(k_attn_merge<64>, dim3(M, a.hq), dim3(64 * kMergeWaves), s, a, nslots);
  return hipErrorInvalidValue;
}

template <class KT, int HD>
static hipError_t launch_hd(const AttnArgs& a, dim3 grid, hipStream_t s) {
  return launch_k(k_attn<KT, HD>, grid, dim3(64 * kAttnWaves), s, a);
}

hipError_t launch_attn(int dtype, int hd, const AttnArgs& a, dim3 grid, hipStream_t s) {
  if (dtype == 2) {
    if (hd == 128) return launch_hd<fp8_t, 128>(a, grid, s);
    if (hd == 64) return launch_hd<fp8_t, 64>(a, grid, s);
  } else if (dtype == 1) {
    if (hd == 128) return launch_hd<bf16_t, 128>(a, grid, s);
    if (hd == 64) return launch_hd<bf16_t, 64>(a, grid, s);
  } else {
    if (hd == 128) return launch_hd<float, 128>(a, grid, s);
    if (hd == 64) return launch_hd<float, 64>(a, grid, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace laser
