// Single-row (decode) attention unit, shared by the standalone decode
// attention kernel and the persistent decode-layer kernel.
//
// A unit is one key range (a "split" of dec_split_keys keys) of one row r and
// one key/value head g; the group's G query heads are the 32 MFMA columns
// (G <= 8 valid), so the keys and values of the head are read once for the
// whole group.  Each of the four waves takes one tile of the range; its K and
// V fragments come straight from memory into registers in MFMA layout (no
// LDS), and the four partial softmax states are merged through LDS.  A row
// with one split writes its output directly; otherwise every split publishes
// its state and the last split of (r, g) to arrive merges them in split order.
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
// block of 256 threads.  DEV: q, K/V and the output are shared with other
// blocks of the same launch (device-scope accesses).
template <int DH, bool DEV>
__device__ __forceinline__ void decode_attn_unit(const DecodeAttnArgs& a, int item, int g, DecodeSmem<DH>& sm) {
  constexpr int TK = (DH == 64) ? 64 : 32;     // keys per tile
  static_assert(TK * 4 == (DH == 64 ? 256 : 128), "a split is one tile per wave");
  constexpr int NST = TK / 32;                 // 32-key score subtiles
  constexpr int NKB = DH / 16;                 // 16-wide K steps of q.k
  constexpr int NDS = DH / 32;                 // output subtiles along dh
  constexpr int NPB = TK / 16;                 // 16-key P.V steps
  auto& red_m = sm.red_m;
  auto& red_l = sm.red_l;
  auto& red_o = sm.red_o;
  int& last = sm.last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 31, fh = lane >> 5;
  const DecItem it = a.items[item];
  const int t = it.t, n_keys = it.n_keys, split = it.split, n_split = it.n_split;
  const int G = a.hq / a.hkv;
  const int kv0 = split * 4 * TK + wave * TK;  // this wave's tile
  const int qh = min(fr, G - 1);  // query head of this lane's column (padding lanes repeat the last)
  const int64_t kbase = it.kbase + int64_t(g) * DH;
  const int64_t vbase = it.vbase + int64_t(g) * DH * a.v_stride;
  const int kstride = a.hkv * DH;

  float m_run = -INFINITY, l_run = 0.0f;
  f32x16 o[NDS];
#pragma unroll
  for (int i = 0; i < NDS; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[i][e] = 0.0f;

  if (kv0 < n_keys) {
    // K rows (A operand of S^T = K Q^T, rows permuted by perm32) and V^T rows
    // (A operand of O^T = V^T P^T); all loads of the tile are issued first.
    u32x4 kf[NST][NKB], vf[NDS][NPB], qf[NKB];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      const int key = kv0 + 32 * st + perm32(fr);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
        kf[st][kb] = ld_u32x4<DEV>(a.kstore + kbase + int64_t(key) * kstride + kb * 16 + fh * 8);
    }
#pragma unroll
    for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb)
        vf[ds][pb] = ld_u32x4<DEV>(a.vstore + vbase + int64_t(ds * 32 + fr) * a.v_stride + kv0 + 16 * pb + 8 * fh);
    {
      const uint16_t* qp = a.q + (int64_t(t) * a.hq + g * G + qh) * DH + fh * 8;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) qf[kb] = ld_u32x4<DEV>(qp + kb * 16);
    }
    // Values past the last key: P is 0 there; keep 0 * garbage out.
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int key = kv0 + 16 * pb + 8 * fh;
      if (key + 8 > n_keys) {
#pragma unroll
        for (int ds = 0; ds < NDS; ++ds)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t lo_ok = (key + 2 * e < n_keys) ? 0x0000ffffu : 0u;
            const uint32_t hi_ok = (key + 2 * e + 1 < n_keys) ? 0xffff0000u : 0u;
            vf[ds][pb][e] &= (lo_ok | hi_ok);
          }
      }
    }

    f32x16 sc[NST];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[st][e] = 0.0f;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) sc[st] = mfma32(kf[st][kb], qf[kb], sc[st]);
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
    m_run = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float psum = 0.0f;
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = exp2f(sc[st][e] - m_run);
        sc[st][e] = p;
        psum += p;
      }
    l_run = psum;
    u32x4 pf[NPB];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int st = pb >> 1, r0 = 8 * (pb & 1);
#pragma unroll
      for (int e = 0; e < 4; ++e) pf[pb][e] = pack2h(sc[st][r0 + 2 * e], sc[st][r0 + 2 * e + 1]);
    }
#pragma unroll
    for (int i = 0; i < NDS; ++i)
#pragma unroll
      for (int pb = 0; pb < NPB; ++pb) o[i] = mfma32(vf[i][pb], pf[pb], o[i]);
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
      st_u16<DEV>(a.o + int64_t(t) * a.hq * DH + (g * G + q) * DH + d, f2h(num / den));
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
    st_u16<DEV>(a.o + int64_t(t) * a.hq * DH + (g * G + q) * DH + (idx % DH), f2h(num / den));
  }
}

}  // namespace decode
}  // namespace hs
