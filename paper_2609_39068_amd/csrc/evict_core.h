// H2O retention and in-place compaction of one unit (Appendix A.3, eq.
// background-h2o-retention; Section 3.1: eviction updates the retained-slot
// mapping and the context length, then releases the discarded slots), run by
// one work-group of NT threads.  Shared by the eviction kernel and by the
// epilogue of the attention kernels (se_decode_step_h2o).
//
// Keys are integers so that selection never compares floats: a slot's keep key
// is (order-preserving bits of its score) << 32 | (0xFFFFFFFF - order-preserving
// bits of its position); larger keeps first, so equal scores keep the lower
// position.
//   * Window: the min(recent, budget) largest positions.  When the recent
//     positions are contiguous (every decode step after the first) it is the
//     positions above max - w; otherwise a radix selection over positions.
//   * One slot over budget: the victim is the candidate with the smallest keep
//     key, found by one block reduction.
//   * Otherwise: radix selection of the budget - |W| largest keep keys.
//   * Compaction: evicted slots below the budget (ascending) are the holes, kept
//     slots at or above it (ascending) are the movers; mover k fills hole k with
//     its key row, value row, position and score.  Sources and destinations are
//     disjoint, so every mover copies independently.
#pragma once

#include <climits>

#include "se_common.h"

namespace se {

constexpr int kMaxBudget = 8192;

struct EvictJob {
  uint16_t* kv;
  int32_t* pos_pool;
  float* score_pool;
  const int32_t* bt;  // the unit's block-table row
  int32_t* lengths;
  int64_t num_pages;
  int32_t unit;
  int32_t L;          // resident slots (read by the caller)
  int32_t budget;
  int32_t recent;
  int32_t max_len;
  int32_t max_pages;
  int32_t* freed_pages;
  int32_t freed_stride;
  int32_t* freed_count;
  int32_t* dev_err;
};

// LDS the caller provides.
template <int NT>
struct EvictScratch {
  int* holes;                    // kMaxBudget
  unsigned* hist;                // 256
  int* scan;                     // NT/64 + 1
  int* bcast;                    // 4
  int* red_i;                    // NT/64
  unsigned long long* red_u64;   // NT/64
};

#define SE_EVICT_SCRATCH(NT, name)                   \
  __shared__ int name##_holes[kMaxBudget];           \
  __shared__ unsigned name##_hist[256];              \
  __shared__ int name##_scan[(NT) / kWave + 1];      \
  __shared__ int name##_bcast[4];                    \
  __shared__ int name##_red_i[(NT) / kWave];         \
  __shared__ unsigned long long name##_red_u64[(NT) / kWave]; \
  const EvictScratch<NT> name{name##_holes, name##_hist, name##_scan, name##_bcast, name##_red_i, name##_red_u64}

__device__ __forceinline__ uint32_t pos_key(int32_t pos) { return (uint32_t)pos ^ 0x80000000u; }

// Calls fn(s, pos, score) for the slots s = lo + tid + k*NT in [lo, hi) of this
// thread, with the positions and scores of BATCH slots loaded before any is
// used, so the loads of a batch overlap instead of each waiting in turn.
template <int NT, int BATCH, typename Fn>
__device__ __forceinline__ void for_slots(const EvictJob& p, int lo, int hi, Fn fn) {
  for (int b = lo + (int)threadIdx.x; b < hi; b += NT * BATCH) {
    int32_t pos[BATCH];
    float u[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int s = b + k * NT;
      if (s < hi) {
        const size_t a = (size_t)p.bt[s >> 4] * kPage + (s & (kPage - 1));
        pos[k] = p.pos_pool[a];
        u[k] = p.score_pool[a];
      }
    }
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int s = b + k * NT;
      if (s < hi) fn(s, pos[k], u[k]);
    }
  }
}

// The same over this thread's contiguous run [lo + tid*R, lo + (tid+1)*R) of
// [lo, hi), in slot order (for rank assignments after one block scan).
template <int NT, int BATCH, typename Fn>
__device__ __forceinline__ void for_run(const EvictJob& p, int lo, int hi, Fn fn) {
  const int R = (hi - lo + NT - 1) / NT;
  const int r0 = lo + (int)threadIdx.x * R;
  const int r1 = min(hi, r0 + R);
  for (int b = r0; b < r1; b += BATCH) {
    int32_t pos[BATCH];
    float u[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int s = b + k;
      if (s < r1) {
        const size_t a = (size_t)p.bt[s >> 4] * kPage + (s & (kPage - 1));
        pos[k] = p.pos_pool[a];
        u[k] = p.score_pool[a];
      }
    }
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int s = b + k;
      if (s < r1) fn(s, pos[k], u[k]);
    }
  }
}

// Radix selection (8-bit digits, most significant first) of the k largest keys
// among the slots for which cand(pos, score) holds; on return an item is among
// them iff (key & *mask) >= *prefix (keys are distinct: positions are).
template <int NT, typename KeyT, typename KeyFn, typename CandFn>
__device__ __forceinline__ void radix_top_slots(const EvictJob& p, int L, int k, KeyFn key_of, CandFn cand,
                                const EvictScratch<NT>& sc, KeyT* prefix_out, KeyT* mask_out) {
  static_assert(NT >= 256 && NT % kWave == 0, "threads 0..255 own one bin each");
  const int tid = threadIdx.x;
  KeyT prefix = 0, mask = 0;
  for (int shift = (int)sizeof(KeyT) * 8 - 8; shift >= 0; shift -= 8) {
    if (tid < 256) sc.hist[tid] = 0;
    __syncthreads();
    for_slots<NT, 8>(p, 0, L, [&](int, int32_t pos, float u) {
      if (!cand(pos, u)) return;
      const KeyT key = key_of(pos, u);
      if ((key & mask) == prefix) atomicAdd(&sc.hist[(unsigned)(key >> shift) & 255u], 1u);
    });
    __syncthreads();
    const int v = tid < 256 ? (int)sc.hist[255 - tid] : 0;  // thread t counts digit 255 - t
    int total;
    const int excl = block_exclusive_scan<NT>(v, sc.scan, &total);
    if (v > 0 && excl < k && excl + v >= k) {
      sc.bcast[0] = 255 - tid;
      sc.bcast[1] = excl;
      sc.bcast[2] = v;
    }
    __syncthreads();
    const int d = sc.bcast[0];
    k -= sc.bcast[1];
    const int cnt = sc.bcast[2];
    __syncthreads();
    prefix |= (KeyT)d << shift;
    mask |= (KeyT)0xFF << shift;
    if (cnt == k) break;
  }
  *prefix_out = prefix;
  *mask_out = mask;
}

template <int NT, int D>
__device__ __forceinline__ void evict_unit(const EvictJob& p, const EvictScratch<NT>& sc) {
  const int tid = threadIdx.x;
  const int unit = p.unit;
  const int L = p.L;
  const int B = p.budget;
  auto fail = [&](uint32_t bit) {
    if (tid == 0) {
      set_error(p.dev_err, bit);
      if (p.freed_count != nullptr) p.freed_count[unit] = 0;
    }
  };
  if (L <= B) {
    if (tid == 0 && p.freed_count != nullptr) p.freed_count[unit] = 0;
    return;
  }
  if (L > p.max_len || L > p.max_pages * kPage) {
    fail(SE_DEVERR_BAD_LENGTH);
    return;
  }
  const int32_t* bt = p.bt;
  const int n_pages = ceil_div_dev(L, kPage);
  {
    int badp = 0;
    for (int i = tid; i < n_pages; i += NT) {
      const int ph = bt[i];
      badp |= (ph < 0 || (int64_t)ph >= p.num_pages);
    }
    badp = block_reduce<NT>(badp, sc.red_i, [](int a, int b) { return a | b; });
    if (badp) {
      fail(SE_DEVERR_BAD_PAGE);
      return;
    }
  }
  auto keep_key = [](int32_t pos, float u) -> uint64_t {
    return ((uint64_t)float_key(u) << 32) | (uint64_t)(0xFFFFFFFFu - pos_key(pos));
  };

  // ---- window W: slots with pos_key >= wthr (none when w == 0)
  const int w = min(p.recent, B);
  uint32_t wthr = 0xFFFFFFFFu;
  const bool wnone = (w == 0);
  if (!wnone) {
    int pmax = INT_MIN;
    for_slots<NT, 8>(p, 0, L, [&](int, int32_t pos, float) { pmax = max(pmax, pos); });
    pmax = block_reduce<NT>(pmax, sc.red_i, [](int a, int b) { return a > b ? a : b; });
    const int64_t lo = (int64_t)pmax - w;  // window = pos > lo when contiguous
    int cnt = 0;
    for_slots<NT, 8>(p, 0, L, [&](int, int32_t pos, float) { cnt += ((int64_t)pos > lo) ? 1 : 0; });
    cnt = block_reduce<NT>(cnt, sc.red_i, [](int a, int b) { return a + b; });
    if (cnt == w) {
      wthr = pos_key((int32_t)(lo + 1));
    } else {
      uint32_t pre, msk;
      radix_top_slots<NT, uint32_t>(
          p, L, w, [](int32_t pos, float) { return pos_key(pos); }, [](int32_t, float) { return true; }, sc,
          &pre, &msk);
      wthr = pre;  // keys are distinct positions: the selection is key >= pre
    }
  }
  auto in_window = [&](int32_t pos) -> bool { return !wnone && pos_key(pos) >= wthr; };

  const int need = B - w;      // candidates to keep
  const int n_evict = L - B;   // slots to drop
  uint64_t kprefix = 0, kmask = 0;
  int victim = -1;
  if (need == 0) {
    // keep the window only
  } else if (n_evict == 1) {
    if (tid == 0) sc.bcast[3] = -1;
    __syncthreads();
    uint64_t best = ~0ull;
    int bslot = -1;
    for_slots<NT, 8>(p, 0, L, [&](int s, int32_t pos, float u) {
      if (in_window(pos)) return;
      const uint64_t k = keep_key(pos, u);
      if (k < best) {
        best = k;
        bslot = s;
      }
    });
    const unsigned long long kmin = block_reduce<NT>((unsigned long long)best, sc.red_u64,
        [](unsigned long long a, unsigned long long b) { return a < b ? a : b; });
    if (best == kmin && bslot >= 0) sc.bcast[3] = bslot;  // keys are distinct
    __syncthreads();
    victim = sc.bcast[3];
    __syncthreads();
    if (victim < 0 || victim >= L) {  // no candidate outside the window: repeated positions
      fail(SE_DEVERR_BAD_POSITIONS);
      return;
    }
  } else {
    radix_top_slots<NT, uint64_t>(
        p, L, need, keep_key, [&](int32_t pos, float) { return !in_window(pos); }, sc, &kprefix, &kmask);
  }
  auto keep = [&](int s, int32_t pos, float u) -> bool {
    if (in_window(pos)) return true;
    if (need == 0) return false;
    if (victim >= 0) return s != victim;
    return (keep_key(pos, u) & kmask) >= kprefix;
  };

  // ---- the retained set must hold exactly B slots (distinct positions)
  int kept = 0;
  for_slots<NT, 8>(p, 0, L, [&](int s, int32_t pos, float u) { kept += keep(s, pos, u) ? 1 : 0; });
  kept = block_reduce<NT>(kept, sc.red_i, [](int a, int b) { return a + b; });
  if (kept != B) {
    fail(SE_DEVERR_BAD_POSITIONS);
    return;
  }

  // ---- compaction
  auto move_slot = [&](int src, int dst, int32_t pos, float u) {
    const uint4* ks = reinterpret_cast<const uint4*>(p.kv + (size_t)bt[src >> 4] * 2 * kPage * D +
                                                     (src & 15) * D);
    uint4* kd = reinterpret_cast<uint4*>(p.kv + (size_t)bt[dst >> 4] * 2 * kPage * D + (dst & 15) * D);
    constexpr int R4 = D / 8;  // 16-byte chunks per row; the value row is one block further
    for (int i = 0; i < R4; i += 2) {  // two chunks of each row in flight
      const uint4 k0 = ks[i], k1 = ks[i + 1];
      const uint4 v0 = ks[i + kPage * R4], v1 = ks[i + 1 + kPage * R4];
      kd[i] = k0;
      kd[i + 1] = k1;
      kd[i + kPage * R4] = v0;
      kd[i + 1 + kPage * R4] = v1;
    }
    const size_t ad = (size_t)bt[dst >> 4] * kPage + (dst & (kPage - 1));
    p.pos_pool[ad] = pos;
    p.score_pool[ad] = u;
  };

  if (victim >= 0) {
    if (tid == 0 && victim != L - 1) {
      const size_t a = (size_t)bt[(L - 1) >> 4] * kPage + ((L - 1) & (kPage - 1));
      move_slot(L - 1, victim, p.pos_pool[a], p.score_pool[a]);
    }
  } else {
    // holes: evicted slots below B, ranked in slot order by one block scan
    int nh = 0;
    for_run<NT, 8>(p, 0, B, [&](int s, int32_t pos, float u) { nh += keep(s, pos, u) ? 0 : 1; });
    int total;
    int rank = block_exclusive_scan<NT>(nh, sc.scan, &total);
    for_run<NT, 8>(p, 0, B, [&](int s, int32_t pos, float u) {
      if (!keep(s, pos, u)) sc.holes[rank++] = s;
    });
    __syncthreads();
    // movers: kept slots at or above B, in slot order, fill the holes in order
    int nm = 0;
    for_run<NT, 8>(p, B, L, [&](int s, int32_t pos, float u) { nm += keep(s, pos, u) ? 1 : 0; });
    rank = block_exclusive_scan<NT>(nm, sc.scan, &total);
    for_run<NT, 8>(p, B, L, [&](int s, int32_t pos, float u) {
      if (keep(s, pos, u)) move_slot(s, sc.holes[rank++], pos, u);
    });
  }

  // ---- release: pages ceil(B/16) .. ceil(L/16)-1 hold nothing now
  const int f0 = ceil_div_dev(B, kPage);
  const int nf = n_pages - f0;
  if (p.freed_pages != nullptr)
    for (int i = tid; i < nf; i += NT) p.freed_pages[(size_t)unit * p.freed_stride + i] = bt[f0 + i];
  if (tid == 0) {
    if (p.freed_count != nullptr) p.freed_count[unit] = nf;
    p.lengths[unit] = B;
  }
}

}  // namespace se
