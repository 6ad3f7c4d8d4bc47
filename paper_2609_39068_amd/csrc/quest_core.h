// Quest page bound of one unit in one work-group (Appendix A.3, eq.
// background-quest-score), shared by the one-kernel selection and by the
// attention kernel's fused selection.
#pragma once

#include "se_common.h"

namespace se {

// Set bits of a wavefront mask below this lane.
__device__ __forceinline__ int lane_prefix_count(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

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

// Lane layout of the page bound: LPP lanes share one page, each with D / LPP
// channels of its minimum and maximum rows (16-byte loads) and of the G query
// rows' positive and negative halves, which take G * D / LPP registers: 8 lanes
// per page, 16 when that would exceed 64 registers (G = 8 at D = 128).
template <int D, int G>
struct BoundLanes {
  static constexpr int LPP = G * D > 512 ? 16 : 8;
  static constexpr int CH = D / LPP;  // channels per lane
  static constexpr int CW = CH / 2;   // bf16 pairs per lane
  static constexpr int C4 = CW / 4;   // 16-byte loads per lane per row
  static_assert(C4 >= 1 && G * CW * 2 <= 64, "bound lane layout");
};

// The lane's channels of the G query rows, split into q+ and q- halves.
template <int D, int G>
__device__ __forceinline__ void bound_query(const uint16_t* q_unit, int g, uint32_t (&qp)[G][BoundLanes<D, G>::CW],
                                            uint32_t (&qn)[G][BoundLanes<D, G>::CW]) {
  using BL = BoundLanes<D, G>;
  const uint16_t* qb = q_unit + g * BL::CH;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const uint4* src = reinterpret_cast<const uint4*>(qb + (size_t)h * D);
#pragma unroll
    for (int i = 0; i < BL::C4; ++i) {
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

// One page's bound (before the scale), the maximum over the G rows of
// q+ . M + q- . m, reduced over the page's LPP lanes (every lane gets it).
template <int D, int G>
__device__ __forceinline__ float page_bound(const uint32_t (&qp)[G][BoundLanes<D, G>::CW],
                                            const uint32_t (&qn)[G][BoundLanes<D, G>::CW],
                                            const uint4 (&mn)[BoundLanes<D, G>::C4],
                                            const uint4 (&mx)[BoundLanes<D, G>::C4]) {
  using BL = BoundLanes<D, G>;
  float acc[G];
#pragma unroll
  for (int h = 0; h < G; ++h) acc[h] = 0.f;
#pragma unroll
  for (int i = 0; i < BL::C4; ++i) {
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
    if constexpr (BL::LPP == 16) a += shfl_xor_f(a, 8);
    best = fmaxf(best, a);
  }
  return best;
}

// Adds one digit per lane (kNoDigit: none) to an LDS histogram.  When every
// lane with a digit has the same one (the common case in a radix selection's
// first passes, whose digits are sign and exponent bits) one lane adds the
// count, instead of 64 atomics on one LDS word.  All 64 lanes must be active.
constexpr uint32_t kNoDigit = 0xFFFFFFFFu;
__device__ __forceinline__ void hist_add_wave(unsigned* hist, uint32_t dg) {
  const uint64_t valid = __ballot(dg != kNoDigit);
  if (valid == 0) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int fl = __builtin_ctzll(valid);
  const uint32_t d0 = __builtin_amdgcn_readlane(dg, fl);
  if (__ballot(dg == d0) == valid) {
    if (lane == fl) atomicAdd(&hist[d0], (unsigned)__popcll(valid));
  } else if (dg != kNoDigit) {
    atomicAdd(&hist[dg], 1u);
  }
}

// Page bounds (eq. background-quest-score) of one unit's candidate pages [0, n)
// by NT threads, LPP lanes per page, into lds_sc (and scores_out when not
// null).  q_unit: the unit's G query rows; lds_bt: its block-table row (-1 for
// an entry outside the pool).  Every iteration's loads are issued before the
// previous page is reduced.  With hist0 (256 zeroed bins), the scores' first
// radix digits (unit_topk's first pass) are counted on the way; with hist1
// (256 zeroed bins), their second digits too, over every score (unit_topk's
// second pass when every score shares the first digit, as page bounds of one
// unit usually do: they lie within a factor of two of each other).
template <int NT, int D, int G>
__device__ __forceinline__ void unit_bounds(const uint16_t* meta_pool, const uint16_t* q_unit, float scale, int n,
                                            const int* lds_bt, float* lds_sc, float* scores_out, unsigned* hist0,
                                            unsigned* hist1) {
  using BL = BoundLanes<D, G>;
  constexpr int CH = BL::CH, CW = BL::CW, C4 = BL::C4, LPP = BL::LPP;
  constexpr int SLOTS = NT / LPP;
  const int lane = threadIdx.x & 63;
  const int g = lane & (LPP - 1);
  const int slot = threadIdx.x / LPP;
  uint32_t qp[G][CW], qn[G][CW];
  bound_query<D, G>(q_unit, g, qp, qn);
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
    const float best = page_bound<D, G>(qp, qn, mn, mx);
    uint32_t dg = kNoDigit, dg1 = kNoDigit;
    if (b < n && g == 0) {
      const float sc = lds_bt[b] >= 0 ? best * scale : -INFINITY;
      lds_sc[b] = sc;
      if (scores_out != nullptr) scores_out[b] = sc;
      dg = float_key(sc) >> 24;
      dg1 = (float_key(sc) >> 16) & 255u;
    }
    if (hist0 != nullptr) hist_add_wave(hist0, dg);
    if (hist1 != nullptr) hist_add_wave(hist1, dg1);
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
// the n scores in lds_sc, by NT threads; emit(r, b) is called for each rank r
// < top_k with the page index b of that rank (-1 past the selection).  Radix
// selection (8-bit digits, most significant first) on order-preserving keys:
// every wavefront adds its keys to an LDS histogram (hist_add_wave), then
// wavefront 0 alone scans the 256 bins, picks the digit and clears the bins.
// With counted, the first pass's histogram is already in hist (unit_bounds
// counts it, and the caller has synchronised); else hist is cleared here.
// pre2 (or null): the second digits of all n keys, counted the same way; it
// is the second pass's histogram when every key has the first pass's digit.
// Then every wavefront takes a contiguous range of indices: it counts its keys
// above the threshold and its keys equal to it, the counts of the ranges
// before it give its output offset, and it emits its selected indices in
// ascending order (keys above the threshold, and the lowest-indexed ones equal
// to it until top_k are taken).
template <int NT, typename Emit>
__device__ __forceinline__ void unit_topk(int n, int top_k, const float* lds_sc, Emit emit, unsigned* hist,
                                          unsigned* pre2, int* bcast, bool counted) {
  constexpr int NW = NT / kWave;
  static_assert(NT >= 256 && NT % kWave == 0, "threads 0..255 clear one bin each");
  static_assert(2 * NW <= 256, "per-wavefront counts live in the histogram");
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const bool w0 = tid < kWave;
  if (n <= top_k) {
    for (int i = tid; i < top_k; i += NT) emit(i, i < n ? i : -1);
    return;
  }
  uint32_t prefix = 0, mask = 0;
  int k = top_k;
  if (!counted) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
  }
  bool have2 = false;  // pre2 is the second pass's histogram
  for (int shift = 24; shift >= 0; shift -= 8) {
    unsigned* const h = have2 && shift == 16 ? pre2 : hist;
    if ((shift < 24 || !counted) && h == hist) {
      for (int i0 = wave * kWave; i0 < n; i0 += NT) {  // wave-uniform trip count
        const int i = i0 + lane;
        uint32_t dg = kNoDigit;
        if (i < n) {
          const uint32_t key = float_key(lds_sc[i]);
          if ((key & mask) == prefix) dg = (key >> shift) & 255u;
        }
        hist_add_wave(hist, dg);
      }
      __syncthreads();
    }
    if (w0) {
      // lane l holds digits 255-4l .. 252-4l (descending); inclusive prefix over lanes
      int c[4], s4 = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = (int)h[255 - 4 * lane - j];
        s4 += c[j];
      }
      int incl = s4;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
      }
      int run = incl - s4;  // keys in higher digits than this lane's first
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (c[j] > 0 && run < k && run + c[j] >= k) {
          bcast[0] = 255 - 4 * lane - j;
          bcast[1] = run;
          bcast[2] = c[j];
        }
        run += c[j];
        h[255 - 4 * lane - j] = 0;  // cleared for a later pass
      }
    }
    __syncthreads();
    const int d = bcast[0];
    k -= bcast[1];
    const int cnt = bcast[2];
    prefix |= (uint32_t)d << shift;
    mask |= 0xFFu << shift;
    if (cnt == k) break;
    // every key has the first digit: the precounted second digits are exact
    have2 = shift == 24 && pre2 != nullptr && cnt == n;
  }
  // k keys equal to the threshold class (under mask) are taken, lowest index
  // first.  Wavefront w owns indices [w * span, (w + 1) * span).
  const int span = (n + NW * kWave - 1) / (NW * kWave) * kWave;
  const int beg = wave * span, end = min(n, beg + span);
  auto classify = [&](int b, bool& above, bool& eq) {
    const uint32_t km = b < end ? (float_key(lds_sc[b]) & mask) : 0u;
    above = b < end && km > prefix;
    eq = b < end && km == prefix;
  };
  int n_above = 0, n_eq = 0;
  for (int b0 = beg; b0 < end; b0 += kWave) {
    bool above, eq;
    classify(b0 + lane, above, eq);
    n_above += __popcll(__ballot(above));
    n_eq += __popcll(__ballot(eq));
  }
  if (lane == 0) {
    hist[wave] = (unsigned)n_above;  // the histogram is free after the last pass's barrier
    hist[NW + wave] = (unsigned)n_eq;
  }
  __syncthreads();
  int taken_above = 0, eq_seen = 0;  // in the ranges before this wavefront's
  for (int v = 0; v < wave; ++v) {
    taken_above += (int)hist[v];
    eq_seen += (int)hist[NW + v];
  }
  for (int b0 = beg; b0 < end; b0 += kWave) {
    const int b = b0 + lane;
    bool above, eq;
    classify(b, above, eq);
    const uint64_t am = __ballot(above), eqm = __ballot(eq);
    const int eq_rank = eq_seen + lane_prefix_count(eqm);
    if (above || (eq && eq_rank < k)) {
      // output rank: the kept keys at lower indices
      emit(taken_above + lane_prefix_count(am) + min(eq_rank, k), b);
    }
    taken_above += __popcll(am);
    eq_seen += __popcll(eqm);
  }
}

}  // namespace se
