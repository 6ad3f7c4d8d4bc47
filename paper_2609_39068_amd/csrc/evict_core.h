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

template <int NT, int D>
__device__ void evict_unit(const EvictJob& p, const EvictScratch<NT>& sc) {
  const int tid = threadIdx.x;
  const int unit = p.unit;
  const int L = p.L;
  const int B = p.budget;
  if (L <= B) {
    if (tid == 0 && p.freed_count != nullptr) p.freed_count[unit] = 0;
    return;
  }
  if (L > p.max_len || L > p.max_pages * kPage) {
    if (tid == 0) {
      set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
      if (p.freed_count != nullptr) p.freed_count[unit] = 0;
    }
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
      if (tid == 0) {
        set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
        if (p.freed_count != nullptr) p.freed_count[unit] = 0;
      }
      return;
    }
  }
  auto addr = [&](int s) -> size_t { return (size_t)bt[s >> 4] * kPage + (s & (kPage - 1)); };
  auto pos_of = [&](int s) -> int32_t { return p.pos_pool[addr(s)]; };
  auto keep_key = [&](int s) -> unsigned long long {
    const size_t a = addr(s);
    return ((unsigned long long)float_key(p.score_pool[a]) << 32) |
           (unsigned long long)(0xFFFFFFFFu - pos_key(p.pos_pool[a]));
  };

  // ---- window W: slots with pos_key >= wthr (none when w == 0)
  const int w = min(p.recent, B);
  uint32_t wthr = 0xFFFFFFFFu;
  bool wnone = (w == 0);
  if (!wnone) {
    int pmax = INT_MIN;
    for (int s = tid; s < L; s += NT) pmax = max(pmax, pos_of(s));
    pmax = block_reduce<NT>(pmax, sc.red_i, [](int a, int b) { return a > b ? a : b; });
    const int64_t lo = (int64_t)pmax - w;  // window = pos > lo when contiguous
    int cnt = 0;
    for (int s = tid; s < L; s += NT) cnt += ((int64_t)pos_of(s) > lo);
    cnt = block_reduce<NT>(cnt, sc.red_i, [](int a, int b) { return a + b; });
    if (cnt == w) {
      wthr = pos_key((int32_t)(lo + 1));
    } else {
      uint32_t pre, msk;
      int krest;
      radix_select_top<NT, uint32_t>(
          L, w, [&](int s) { return pos_key(pos_of(s)); }, [](int) { return true; }, &pre, &msk,
          &krest, sc.hist, sc.scan, sc.bcast);
      wthr = pre;  // keys are distinct positions: the selection is key >= pre
    }
  }
  auto in_window = [&](int s) -> bool { return !wnone && pos_key(pos_of(s)) >= wthr; };

  const int need = B - w;      // candidates to keep
  const int n_evict = L - B;   // slots to drop
  uint64_t kprefix = 0, kmask = 0;
  int victim = -1;
  if (need == 0) {
    // keep the window only
  } else if (n_evict == 1) {
    if (tid == 0) sc.bcast[3] = -1;
    __syncthreads();
    unsigned long long best = ~0ull;
    int bslot = -1;
    for (int s = tid; s < L; s += NT) {
      if (in_window(s)) continue;
      const unsigned long long k = keep_key(s);
      if (k < best) {
        best = k;
        bslot = s;
      }
    }
    unsigned long long packed_min = block_reduce<NT>(best, sc.red_u64, [](unsigned long long a,
                                                                       unsigned long long b) {
      return a < b ? a : b;
    });
    // recover the slot holding the minimum key (keys are distinct)
    if (best == packed_min && bslot >= 0) sc.bcast[3] = bslot;
    __syncthreads();
    victim = sc.bcast[3];
    __syncthreads();
    if (victim < 0 || victim >= L) {  // no candidate outside the window: repeated positions
      if (tid == 0) {
        set_error(p.dev_err, SE_DEVERR_BAD_POSITIONS);
        if (p.freed_count != nullptr) p.freed_count[unit] = 0;
      }
      return;
    }
  } else {
    int krest;
    radix_select_top<NT, uint64_t>(
        L, need, [&](int s) { return (uint64_t)keep_key(s); },
        [&](int s) { return !in_window(s); }, &kprefix, &kmask, &krest, sc.hist, sc.scan, sc.bcast);
  }
  auto keep = [&](int s) -> bool {
    if (in_window(s)) return true;
    if (need == 0) return false;
    if (victim >= 0) return s != victim;
    return ((uint64_t)keep_key(s) & kmask) >= kprefix;
  };

  // ---- the retained set must hold exactly B slots (distinct positions)
  int kept = 0;
  for (int s = tid; s < L; s += NT) kept += keep(s) ? 1 : 0;
  kept = block_reduce<NT>(kept, sc.red_i, [](int a, int b) { return a + b; });
  if (kept != B) {
    if (tid == 0) {
      set_error(p.dev_err, SE_DEVERR_BAD_POSITIONS);
      if (p.freed_count != nullptr) p.freed_count[unit] = 0;
    }
    return;
  }

  // ---- compaction
  auto move_slot = [&](int src, int dst) {
    const size_t as = addr(src), ad = addr(dst);
    const uint4* ks = reinterpret_cast<const uint4*>(p.kv + (size_t)bt[src >> 4] * 2 * kPage * D +
                                                     (src & 15) * D);
    uint4* kd = reinterpret_cast<uint4*>(p.kv + (size_t)bt[dst >> 4] * 2 * kPage * D + (dst & 15) * D);
    constexpr int R4 = D / 8;  // 16-byte chunks per row
#pragma unroll 4
    for (int i = 0; i < R4; ++i) {
      kd[i] = ks[i];
      kd[i + kPage * R4] = ks[i + kPage * R4];  // value row, one block further
    }
    p.pos_pool[ad] = p.pos_pool[as];
    p.score_pool[ad] = p.score_pool[as];
  };

  if (victim >= 0) {
    if (tid == 0 && victim != L - 1) move_slot(L - 1, victim);
  } else {
    int base = 0;
    for (int s0 = 0; s0 < B; s0 += NT) {
      const int s = s0 + tid;
      const int flag = (s < B && !keep(s)) ? 1 : 0;
      int total;
      const int rank = block_exclusive_scan<NT>(flag, sc.scan, &total);
      if (flag) sc.holes[base + rank] = s;
      base += total;
    }
    __syncthreads();
    int mbase = 0;
    for (int s0 = B; s0 < L; s0 += NT) {
      const int s = s0 + tid;
      const int flag = (s < L && keep(s)) ? 1 : 0;
      int total;
      const int rank = block_exclusive_scan<NT>(flag, sc.scan, &total);
      if (flag) move_slot(s, sc.holes[mbase + rank]);
      mbase += total;
    }
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
