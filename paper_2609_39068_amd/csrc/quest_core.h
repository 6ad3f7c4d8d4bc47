// Quest page bound of one unit in one work-group (Appendix A.3, eq.
// background-quest-score), shared by the one-kernel selection and by the
// attention kernel's fused selection.
#pragma once

#include "se_common.h"

namespace se {

// bf16 pair with negative halves zeroed (q+) or non-negative halves zeroed (q-).
__device__ __forceinline__ uint32_t pos_part(uint32_t x) {
  const uint32_t lo = (x & 0x8000u) ? 0u : (x & 0xffffu);
  const uint32_t hi = (x & 0x80000000u) ? 0u : (x & 0xffff0000u);
  return lo | hi;
}
__device__ __forceinline__ uint32_t neg_part(uint32_t x) {
  const uint32_t lo = (x & 0x8000u) ? (x & 0xffffu) : 0u;
  const uint32_t hi = (x & 0x80000000u) ? (x & 0xffff0000u) : 0u;
  return lo | hi;
}

// Page bounds (eq. background-quest-score) of one unit's candidate pages [0, n)
// by NT threads, 8 lanes per page, into lds_sc (and scores_out when not null).
// q_unit: the unit's G query rows; lds_bt: its block-table row (-1 for an entry
// outside the pool).  Every iteration's loads are issued before the previous
// page is reduced.
template <int NT, int D, int G>
__device__ __forceinline__ void unit_bounds(const uint16_t* meta_pool, const uint16_t* q_unit, float scale, int n,
                                            const int* lds_bt, float* lds_sc, float* scores_out) {
  constexpr int CH = D / 8;   // channels per lane
  constexpr int CW = CH / 2;  // bf16 pairs per lane
  constexpr int C4 = CW / 4;  // 16-byte loads per lane per row
  constexpr int SLOTS = NT / 8;
  const int lane = threadIdx.x & 63;
  const int g = lane & 7;
  const int slot = threadIdx.x >> 3;
  uint32_t qp[G][CW], qn[G][CW];
  {
    const uint16_t* qb = q_unit + g * CH;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const uint4* src = reinterpret_cast<const uint4*>(qb + (size_t)h * D);
#pragma unroll
      for (int i = 0; i < C4; ++i) {
        const uint4 t = src[i];
        const uint32_t v[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          qp[h][4 * i + e] = pos_part(v[e]);
          qn[h][4 * i + e] = neg_part(v[e]);
        }
      }
    }
  }
  auto load = [&](int b, uint4 (&mn)[C4], uint4 (&mx)[C4]) {
    const int ph = lds_bt[min(b, n - 1)];
    const uint16_t* meta = meta_pool + (size_t)(ph < 0 ? 0 : ph) * 2 * D + g * CH;
#pragma unroll
    for (int i = 0; i < C4; ++i) {
      mn[i] = reinterpret_cast<const uint4*>(meta)[i];
      mx[i] = reinterpret_cast<const uint4*>(meta + D)[i];
    }
  };
  auto bound = [&](int b, const uint4 (&mn)[C4], const uint4 (&mx)[C4]) {
    float acc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = 0.f;
#pragma unroll
    for (int i = 0; i < C4; ++i) {
      const uint32_t lo[4] = {mn[i].x, mn[i].y, mn[i].z, mn[i].w};
      const uint32_t hi[4] = {mx[i].x, mx[i].y, mx[i].z, mx[i].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          acc[h] = dot2bf16(qp[h][4 * i + e], hi[e], acc[h]);
          acc[h] = dot2bf16(qn[h][4 * i + e], lo[e], acc[h]);
        }
      }
    }
    float best = -INFINITY;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float a = quad_sum(acc[h]);
      a += shfl_xor_f(a, 4);
      best = fmaxf(best, a);
    }
    if (b < n && g == 0) {
      const float sc = lds_bt[b] >= 0 ? best * scale : -INFINITY;
      lds_sc[b] = sc;
      if (scores_out != nullptr) scores_out[b] = sc;
    }
  };
  const int iters = (n + SLOTS - 1) / SLOTS;
  uint4 mnA[C4], mxA[C4], mnB[C4], mxB[C4];
  if (iters > 0) load(slot, mnA, mxA);
  for (int it = 0; it < iters; it += 2) {
    load(slot + (it + 1) * SLOTS, mnB, mxB);
    bound(slot + it * SLOTS, mnA, mxA);
    if (it + 1 >= iters) break;
    load(slot + (it + 2) * SLOTS, mnA, mxA);
    bound(slot + (it + 1) * SLOTS, mnB, mxB);
  }
}

// The top_k pages of one unit by score (ties: lower page index), ascending, from
// the n scores in lds_sc, by NT threads; written to out_g and out_l (either may
// be null), -1 past the selection.  Radix selection on order-preserving keys,
// then the selected indices ranked by block scans.
template <int NT>
__device__ __forceinline__ void unit_topk(int n, int top_k, const float* lds_sc, int32_t* out_g, int32_t* out_l,
                                          unsigned* hist, int* scan_scratch, int* bcast) {
  const int tid = threadIdx.x;
  if (n <= top_k) {
    for (int i = tid; i < top_k; i += NT) {
      const int v = i < n ? i : -1;
      if (out_g != nullptr) out_g[i] = v;
      if (out_l != nullptr) out_l[i] = v;
    }
    return;
  }
  auto key_of = [&](int b) { return float_key(lds_sc[b]); };
  uint32_t prefix, mask;
  int k_rest;
  radix_select_top<NT, uint32_t>(n, top_k, key_of, [](int) { return true; }, &prefix, &mask, &k_rest, hist,
                                 scan_scratch, bcast);
  // keys above the threshold class, then the first k_rest of the class in index order
  int eq_base = 0, out_base = 0;
  for (int b0 = 0; b0 < n; b0 += NT) {
    const int b = b0 + tid;
    uint32_t km = 0;
    if (b < n) km = key_of(b) & mask;
    const int is_eq = (b < n && km == prefix) ? 1 : 0;
    int eq_total;
    const int eq_rank = block_exclusive_scan<NT>(is_eq, scan_scratch, &eq_total);
    const int take = (b < n) && (km > prefix || (is_eq && eq_base + eq_rank < k_rest)) ? 1 : 0;
    int take_total;
    const int rank = block_exclusive_scan<NT>(take, scan_scratch, &take_total);
    if (take) {
      if (out_g != nullptr) out_g[out_base + rank] = b;
      if (out_l != nullptr) out_l[out_base + rank] = b;
    }
    eq_base += eq_total;
    out_base += take_total;
  }
}

}  // namespace se
