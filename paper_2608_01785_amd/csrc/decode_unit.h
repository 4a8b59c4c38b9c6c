// Single-row (decode) attention unit.
//
// A unit is one key range (a "split" of unit_keys keys, inside one page of
// the cache) of one row r and
// one key/value head g; the group's G query heads are the 32 MFMA columns
// (G <= 8 valid), so the keys and values of the head are read once for the
// whole group.  The range is cut into tiles (dec_tile_keys keys); wave w takes
// tiles w, w + 4, w + 8, ... and keeps its own running softmax state over
// them.  A tile's K and V fragments go from memory straight into registers in
// MFMA layout (no LDS), two register sets deep, so the next tile's loads are
// in flight while the current tile is multiplied.  The four waves' states are
// merged through LDS.  A row with one split writes its output directly;
// otherwise every split publishes its state and the last split of (r, g) to
// arrive merges them in split order.
#pragma once

#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {
namespace decode {

constexpr int kUnitThreads = 256;  // threads per block running a unit

template <int DH>
struct DecodeSmem {
  float red_m[4][8], red_l[4][8];
  float red_o[4][DH][9];  // [wave][d][query head], G <= 8
  int last;
};

// One work item (a key range of one row) for one key/value head g, by one
// block of 256 threads.
template <int DH>
__device__ __forceinline__ void decode_attn_unit(const DecodeAttnArgs& a, int item, int g, DecodeSmem<DH>& sm) {
  constexpr int TK = dec_tile_keys(DH);        // keys per tile
  constexpr int NST = TK / 32;                 // 32-key score subtiles
  constexpr int NKB = DH / 16;                 // 16-wide K steps of q.k
  constexpr int NDS = DH / 32;                 // output subtiles along dh
  constexpr int NPB = TK / 16;                 // 16-key P.V steps
  auto& red_m = sm.red_m;
  auto& red_l = sm.red_l;
  auto& red_o = sm.red_o;
  int& last = sm.last;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 31, fh = lane >> 5;
  const DecItem it = a.items[item];
  const int t = it.t, n_keys = it.n_keys, split = it.split, n_split = it.n_split;
  const int G = a.hq / a.hkv;
  const int k_begin = split * a.unit_keys;
  const int n_tiles = (min(n_keys - k_begin, a.unit_keys) + TK - 1) / TK;
  // The range lies in one page (of a slot or the packed buffer): its first
  // key sits at key0 = k_begin rounded down to the page size.
  const int key0 = k_begin - k_begin % a.page_keys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + 3) / 4 : 0;
  const int qh = min(fr, G - 1);  // query head of this lane's column (padding lanes repeat the last)
  const int64_t kbase = it.kbase + int64_t(g) * a.kv_head_stride;
  const int64_t vbase = it.vbase + int64_t(g) * a.kv_head_stride;

  float m_run = -INFINITY, l_run = 0.0f;
  f32x16 o[NDS];
#pragma unroll
  for (int i = 0; i < NDS; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[i][e] = 0.0f;

  u32x4 qf[NKB];
  {
    const uint16_t* qp = a.q + (int64_t(t) * a.hq + g * G + qh) * DH + fh * 8;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) qf[kb] = *reinterpret_cast<const u32x4*>(qp + kb * 16);
  }

  // K rows (A operand of S^T = K Q^T, rows permuted by perm32) and V^T rows
  // (A operand of O^T = V^T P^T) of tile `ti` of the range, through buffer
  // resources based at the range's page and head: per-lane offsets are
  // fixed, the tile moves the scalar offset.  A tile is one 32-key value tile
  // of the cache, and its key rows are contiguous too.  Keys past the last
  // one stay inside the page (ranges are whole tiles of a page whose length
  // is a multiple of 64); their scores are masked below.
  static_assert(TK == kv_tile_keys, "a tile is one value tile of the cache");
  const __amdgpu_buffer_rsrc_t kres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.kstore + kbase), 0, 0x7ffffff0, 0x00020000);
  const __amdgpu_buffer_rsrc_t vres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.vstore + vbase), 0, 0x7ffffff0, 0x00020000);
  const uint32_t k_lane = uint32_t(perm32(fr) * DH * 2 + fh * 16);
  const uint32_t v_lane = uint32_t(fr * TK * 2 + fh * 16);
  constexpr uint32_t v_sub = 32 * TK * 2;  // bytes between 32-dimension subtiles of a value tile
  struct Tile {
    u32x4 k[NST][NKB];
    u32x4 v[NDS][NPB];
  };
  auto load_tile = [&](int ti, Tile& tl) {
    const int kv0 = k_begin + ti * TK - key0;  // key index inside the page
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      const uint32_t so = uint32_t((kv0 + 32 * st) * DH * 2);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
        tl.k[st][kb] = __builtin_amdgcn_raw_buffer_load_b128(kres, k_lane + kb * 32, so, 0);
    }
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb)
        tl.v[ds][pb] = __builtin_amdgcn_raw_buffer_load_b128(vres, v_lane + pb * 32,
                                                             uint32_t(ds) * v_sub + uint32_t(kv0 * DH * 2), 0);
  };
  // Online softmax over this wave's tiles, in the exp2 domain.
  auto compute_tile = [&](int ti, Tile& tl) {
    const int kv0 = k_begin + ti * TK;
    if (kv0 + TK > n_keys) {
      // Values past the last key: P is 0 there; keep 0 * garbage out.
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb) {
        const int key = kv0 + 16 * pb + 8 * fh;
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t lo_ok = (key + 2 * e < n_keys) ? 0x0000ffffu : 0u;
            const uint32_t hi_ok = (key + 2 * e + 1 < n_keys) ? 0xffff0000u : 0u;
            tl.v[ds][pb][e] &= (lo_ok | hi_ok);
          }
      }
    }
    f32x16 sc[NST];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[st][e] = 0.0f;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) sc[st] = mfma32(tl.k[st][kb], qf[kb], sc[st]);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = kv0 + 32 * st + 16 * (e >> 3) + 8 * fh + (e & 7);
        const float v = (key < n_keys) ? sc[st][e] * a.scale_log2 : -INFINITY;
        sc[st][e] = v;
        mx = fmaxf(mx, v);
      }
    // Every tile holds at least one valid key, so m_new is finite.
    const float m_new = fmaxf(m_run, fmaxf(mx, __shfl_xor(mx, 32, 64)));
    const float alpha = exp2f(m_run - m_new);  // 0 on the first tile
    m_run = m_new;
    float psum = 0.0f;
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = exp2f(sc[st][e] - m_new);
        sc[st][e] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
    u32x4 pf[NPB];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int st = pb >> 1, r0 = 8 * (pb & 1);
#pragma unroll
      for (int e = 0; e < 4; ++e) pf[pb][e] = pack2h(sc[st][r0 + 2 * e], sc[st][r0 + 2 * e + 1]);
    }
#pragma unroll
    for (int i = 0; i < NDS; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) o[i][e] *= alpha;
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb) o[i] = mfma32(tl.v[i][pb], pf[pb], o[i]);
    }
  };

  if constexpr (DH == 64) {
    // Two register sets.  The first load is unconditional (a wave without
    // tiles reads tile 0 and discards it); later loads run only for tiles the
    // wave owns, so the compiler's wait counts stay exact.  The scheduling
    // barriers keep each tile's loads ahead of the previous tile's math.
    Tile t0, t1;
    load_tile(my_tiles > 0 ? wave : 0, t0);
    __builtin_amdgcn_sched_barrier(0);
    int i = 0;
    for (; i + 2 < my_tiles; i += 2) {
      load_tile(wave + 4 * (i + 1), t1);
      __builtin_amdgcn_sched_barrier(0);
      compute_tile(wave + 4 * i, t0);
      __builtin_amdgcn_sched_barrier(0);
      load_tile(wave + 4 * (i + 2), t0);
      __builtin_amdgcn_sched_barrier(0);
      compute_tile(wave + 4 * (i + 1), t1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (my_tiles - i == 2) {
      load_tile(wave + 4 * (i + 1), t1);
      __builtin_amdgcn_sched_barrier(0);
      compute_tile(wave + 4 * i, t0);
      __builtin_amdgcn_sched_barrier(0);
      compute_tile(wave + 4 * (i + 1), t1);
    } else if (my_tiles - i == 1) {
      compute_tile(wave + 4 * i, t0);
    }
  } else {
    // head_dim 128: a tile's fragments and the larger output and query
    // registers leave room for one register set; other waves of the CU
    // overlap the loads.
    Tile t0;
    for (int i = 0; i < my_tiles; ++i) {
      load_tile(wave + 4 * i, t0);
      compute_tile(wave + 4 * i, t0);
    }
  }

  // Merge the four waves.  Lane (fr, fh) holds query column fr; both halves
  // share the maximum, each holds part of the sum.  Waves without a tile hold
  // -inf and weigh zero.
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (fh == 0 && fr < 8) {
    red_m[wave][fr] = m_run;
    red_l[wave][fr] = l_tot;
  }
  if (fr < 8) {
#pragma unroll
    for (int i = 0; i < NDS; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) red_o[wave][32 * i + 8 * (e >> 2) + 4 * fh + (e & 3)][fr] = o[i][e];
  }
  __syncthreads();

  const int pf_stride = dec_part_floats(G, DH);
  const int64_t row_item0 = item - split;  // first split of this row
  for (int idx = tid; idx < G * DH; idx += kUnitThreads) {
    const int q = idx / DH, d = idx % DH;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, red_m[w][q]);
    float num = 0.0f, den = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float sc = exp2f(red_m[w][q] - M);
      num += sc * red_o[w][d][q];
      den += sc * red_l[w][q];
    }
    if (n_split == 1) {
      a.o[act_index(t, (g * G + q) * DH + d, a.hq * DH, a.o_k8_rows)] = f2h(num / den);
    } else {
      // Publish (unnormalised output, maximum, sum) with device-scope stores.
      float* st = a.part + (int64_t(item) * a.hkv + g) * pf_stride;
      __hip_atomic_store(st + idx, num, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (d == 0) {
        __hip_atomic_store(st + G * DH + q, M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(st + G * DH + G + q, den, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  if (n_split == 1) return;

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // partial state complete before the arrival count
  __syncthreads();
  if (tid == 0) {
    int32_t* cnt = a.counters + row_item0 * a.hkv + g;
    last = atomicAdd(cnt, 1) == n_split - 1;
    if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!last) return;

  // Last arrival: combine the splits of (r, g) in split order, eight at a
  // time (all loads of a batch in flight), with a running maximum.
  const float* base = a.part + (row_item0 * a.hkv + g) * pf_stride;
  const int64_t split_stride = int64_t(a.hkv) * pf_stride;
  for (int idx = tid; idx < G * DH; idx += kUnitThreads) {
    const int q = idx / DH;
    float M = -INFINITY, num = 0.0f, den = 0.0f;
    for (int sp0 = 0; sp0 < n_split; sp0 += 8) {
      float mv[8], lv[8], ov[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float* st = base + min(sp0 + k, n_split - 1) * split_stride;
        mv[k] = __hip_atomic_load(st + G * DH + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        lv[k] = __hip_atomic_load(st + G * DH + G + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ov[k] = __hip_atomic_load(st + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      float bm = M;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (sp0 + k < n_split) bm = fmaxf(bm, mv[k]);
      const float rescale = exp2f(M - bm);  // M = -inf on the first batch: 0
      num *= rescale;
      den *= rescale;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (sp0 + k < n_split) {
          const float sc = exp2f(mv[k] - bm);
          num += sc * ov[k];
          den += sc * lv[k];
        }
      }
      M = bm;
    }
    a.o[act_index(t, (g * G + q) * DH + idx % DH, a.hq * DH, a.o_k8_rows)] = f2h(num / den);
  }
}

}  // namespace decode
}  // namespace hs
