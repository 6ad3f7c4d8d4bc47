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
  int32_t* moves = nullptr;  // deferred moves: count, then holes, then movers (kMoveListInts ints)
};

// A unit's deferred move list: moves[0] = n, holes at moves[kMoveHoles + r],
// movers at moves[kMoveMovers + r], r < n (slot indices).
constexpr int kMoveHoles = 64;
constexpr int kMoveMovers = kMoveHoles + kMaxBudget;
constexpr int kMoveListInts = kMoveMovers + kMaxBudget;

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

// Arguments of the standalone eviction kernel (one work-group per unit, each
// unit's resident length read from lengths[]), launched by launch_evict.
struct EvictParams {
  uint16_t* kv;
  int32_t* pos_pool;
  float* score_pool;
  const int32_t* block_table;
  int32_t* lengths;
  int64_t num_pages;
  int32_t max_pages;
  int32_t budget;
  int32_t recent;
  int32_t max_len;
  int32_t* freed_pages;
  int32_t freed_stride;
  int32_t* freed_count;
  int32_t* dev_err;
  // When set (kMoveListInts ints per unit), the selection kernel leaves each
  // unit's holes and movers here and a second kernel, several work-groups per
  // unit, moves the rows.
  int32_t* moves = nullptr;
};

// Launches the eviction of every unit (head_dim 64 or 128) on `stream`.
void launch_evict(const EvictParams& p, int num_units, int head_dim, hipStream_t stream);

// The same with the holes array supplied by the caller (kMaxBudget ints of LDS
// that it also uses for something else before the eviction starts).
#define SE_EVICT_SCRATCH_WITH_HOLES(NT, name, holes_ptr) \
  __shared__ unsigned name##_hist[256];                  \
  __shared__ int name##_scan[(NT) / kWave + 1];          \
  __shared__ int name##_bcast[4];                        \
  __shared__ int name##_red_i[(NT) / kWave];             \
  __shared__ unsigned long long name##_red_u64[(NT) / kWave]; \
  const EvictScratch<NT> name{(holes_ptr), name##_hist, name##_scan, name##_bcast, name##_red_i, name##_red_u64}

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

namespace se {

// ---------------------------------------------------------------------------
// Register-resident variant for large units (one work-group of NT threads,
// NT * KPT slots at most, KPT <= 64).  Thread tid owns the slots
// s = k * NT + tid, k < KPT (coalesced reads through the block-table row
// staged in LDS) and holds their order-preserving score bits in registers,
// plus two bit masks over its rows: in the window, and retained.
//   * Window: the positions are held for this phase only -- the newest
//     position, then the rows above newest - w; when that run is not exactly
//     w long, a radix selection over positions gives the threshold.
//   * Selection on the score bits alone (at most four 8-bit radix passes over
//     registers).  Only if scores tie exactly at the threshold are positions
//     needed: the tied candidates with the lowest positions fill what is left
//     (a radix selection over their positions), which is the keep-key order.
//   * Ranking: per (row, wavefront) counts of holes and movers from ballots,
//     one block scan over those counts in slot order, each slot's rank from
//     the scanned base plus its lane's prefix in the ballot; holes and movers
//     are listed in LDS by rank.
//   * Mover r's key and value rows, position and score go to hole r, copied
//     by the whole work-group, one 16-byte chunk per thread, four movers in
//     flight per thread.
// Larger units take evict_unit.
//
// The radix histogram is replicated kHistCopies times (copy = lane mod
// kHistCopies, copies kHistStride words apart so that they sit in different
// banks): lanes of a wavefront that share a digit -- most of them in the first
// pass, where scores of similar magnitude share their top bits -- then update
// different words instead of serialising on one.
constexpr int kHistCopies = 16;
constexpr int kHistStride = 257;

template <int NT, int KPT>
struct WideScratch {
  EvictScratch<NT> base;
  int* movers;      // kMaxBudget
  int* bt;          // NT * KPT / kPage
  int* cnt_h;       // KPT * NT / kWave
  int* cnt_m;       // KPT * NT / kWave
  unsigned* hist;   // kHistCopies * kHistStride
};

#define SE_WIDE_SCRATCH(NT, KPT, name)                          \
  SE_EVICT_SCRATCH(NT, name##_b);                               \
  __shared__ int name##_movers[kMaxBudget];                     \
  __shared__ int name##_bt[(NT) * (KPT) / kPage];               \
  __shared__ int name##_ch[(KPT) * (NT) / kWave];               \
  __shared__ int name##_cm[(KPT) * (NT) / kWave];               \
  __shared__ unsigned name##_hist[kHistCopies * kHistStride];   \
  const WideScratch<NT, KPT> name{name##_b, name##_movers, name##_bt, name##_ch, name##_cm, name##_hist}

__device__ __forceinline__ int lane_prefix(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Values behind an empty asm.  The optimiser would otherwise merge every use
// of a per-row value (a row's slot index k * NT + tid, a row's candidate test)
// into one register per row that stays live -- and spills -- across phases;
// laundered, such values are recomputed in each phase.
__device__ __forceinline__ int opaque_int(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

template <int KPT>
__device__ __forceinline__ void opaque_rows(uint32_t (&fk)[KPT], uint64_t& bits, int& nrow) {
#pragma unroll
  for (int i = 0; i < KPT; ++i) asm volatile("" : "+v"(fk[i]));
  asm volatile("" : "+v"(bits), "+v"(nrow));
}

// Radix selection (8-bit digits) of the k largest score keys among this
// thread's rows i < nrow outside the window (bit clear in win).  Returns the
// prefix; a row is selected iff (key & *mask) >= prefix, except that when the
// last pass ends on a class of exactly equal keys larger than what is left,
// only part of that class belongs to the selection (the caller splits it).
template <int NT, int KPT>
__device__ __forceinline__ uint32_t radix_score_regs(int k, uint32_t (&fk)[KPT], uint64_t win, int nrow,
                                                     const WideScratch<NT, KPT>& ws, uint32_t* mask_out) {
  static_assert(NT >= 256, "threads 0..255 own one bin each");
  const EvictScratch<NT>& sc = ws.base;
  const int tid = threadIdx.x;
  unsigned* const hist = ws.hist + (tid % kHistCopies) * kHistStride;
  uint32_t prefix = 0, mask = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    opaque_rows<KPT>(fk, win, nrow);
    for (int i = tid; i < kHistCopies * kHistStride; i += NT) ws.hist[i] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KPT; ++i)
      if (i < nrow && !((win >> i) & 1) && (fk[i] & mask) == prefix)
        atomicAdd(&hist[(fk[i] >> shift) & 255u], 1u);
    __syncthreads();
    int v = 0;  // thread t counts digit 255 - t over the copies
    if (tid < 256)
#pragma unroll
      for (int c = 0; c < kHistCopies; ++c) v += (int)ws.hist[c * kHistStride + 255 - tid];
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
    prefix |= (uint32_t)d << shift;
    mask |= 0xFFu << shift;
    if (cnt == k) break;
  }
  *mask_out = mask;
  return prefix;
}

template <int NT, int D, int KPT>
__device__ __forceinline__ void evict_unit_wide(const EvictJob& p, const WideScratch<NT, KPT>& ws) {
  static_assert(NT % kWave == 0 && KPT <= 64 && KPT * (NT / kWave) <= NT, "row bits and scan entries");
  constexpr int NW = NT / kWave;
  const EvictScratch<NT>& sc = ws.base;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
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
  if (L > NT * KPT) {
    evict_unit<NT, D>(p, sc);
    return;
  }
  const int n_pages = ceil_div_dev(L, kPage);
  {
    int badp = 0;
    for (int i = tid; i < n_pages; i += NT) {
      const int ph = p.bt[i];
      badp |= (ph < 0 || (int64_t)ph >= p.num_pages);
      ws.bt[i] = ph;
    }
    badp = block_reduce<NT>(badp, sc.red_i, [](int a, int b) { return a | b; });  // also publishes ws.bt
    if (badp) {
      fail(SE_DEVERR_BAD_PAGE);
      return;
    }
  }
  int nrow = (L - tid + NT - 1) / NT;  // rows k with k * NT + tid < L
  auto addr = [&](int s) -> size_t { return (size_t)ws.bt[s >> 4] * kPage + (s & (kPage - 1)); };

  // ---- window W (bit k of win: row k is in it)
  const int w = min(p.recent, B);
  uint64_t win = 0;
  uint32_t wthr = 0xFFFFFFFFu;  // W = slots with pos_key >= wthr
  if (w > 0) {
    int32_t pos[KPT];
    {
      const int t = opaque_int(tid);
#pragma unroll
      for (int k = 0; k < KPT; ++k) pos[k] = p.pos_pool[addr(min(k * NT + t, L - 1))];
    }
    int pmax = INT_MIN;
#pragma unroll
    for (int k = 0; k < KPT; ++k) pmax = max(pmax, pos[k]);  // rows past L repeat slot L - 1
    pmax = block_reduce<NT>(pmax, sc.red_i, [](int a, int b) { return a > b ? a : b; });
    const int64_t lo = (int64_t)pmax - w;  // window = pos > lo when the newest w are contiguous
#pragma unroll
    for (int k = 0; k < KPT; ++k)
      if (k < nrow && (int64_t)pos[k] > lo) win |= 1ull << k;
    const int cnt = block_reduce<NT>((int)__popcll(win), sc.red_i, [](int a, int b) { return a + b; });
    if (cnt == w) {
      wthr = pos_key((int32_t)(lo + 1));
    } else {
      uint32_t pre, msk;
      radix_top_slots<NT, uint32_t>(
          p, L, w, [](int32_t q, float) { return pos_key(q); }, [](int32_t, float) { return true; }, sc, &pre,
          &msk);
      wthr = pre;
      win = 0;
      const int t = opaque_int(tid);
#pragma unroll
      for (int k = 0; k < KPT; ++k)
        if (k < nrow && pos_key(p.pos_pool[addr(k * NT + t)]) >= wthr) win |= 1ull << k;
    }
  }

  // ---- scores: order-preserving bits, one register per row
  uint32_t fk[KPT];
  {
    const int t = opaque_int(tid);
#pragma unroll
    for (int k = 0; k < KPT; ++k) fk[k] = __float_as_uint(p.score_pool[addr(min(k * NT + t, L - 1))]);
#pragma unroll
    for (int k = 0; k < KPT; ++k) fk[k] = float_key(__uint_as_float(fk[k]));
  }

  // ---- selection of the need = B - |W| candidates to keep
  const int need = B - w;
  const int n_evict = L - B;
  uint64_t keep = win;  // bit k: row k is retained
  if (need > 0 && n_evict == 1) {
    // one victim: the smallest score outside the window, the largest position among equal scores
    uint32_t fmin = 0xFFFFFFFFu;
#pragma unroll
    for (int k = 0; k < KPT; ++k)
      if (k < nrow && !((win >> k) & 1)) fmin = min(fmin, fk[k]);
    fmin = block_reduce<NT>(fmin, reinterpret_cast<uint32_t*>(sc.red_i),
                            [](uint32_t a, uint32_t b) { return a < b ? a : b; });
    if (tid == 0) sc.bcast[3] = -1;
    int pbest = INT_MIN, sbest = -1;
    {
      const int t = opaque_int(tid);
#pragma unroll
      for (int k = 0; k < KPT; ++k)
        if (k < nrow && !((win >> k) & 1) && fk[k] == fmin) {
          const int pos = p.pos_pool[addr(k * NT + t)];
          if (sbest < 0 || pos > pbest) {
            pbest = pos;
            sbest = k * NT + t;
          }
        }
    }
    const int pm = block_reduce<NT>(sbest >= 0 ? pbest : INT_MIN, sc.red_i,
                                    [](int a, int b) { return a > b ? a : b; });
    if (sbest >= 0 && pbest == pm) sc.bcast[3] = sbest;  // positions are distinct
    __syncthreads();
    const int victim = sc.bcast[3];
    __syncthreads();
    if (victim < 0 || victim >= L) {  // no candidate outside the window: repeated positions
      fail(SE_DEVERR_BAD_POSITIONS);
      return;
    }
    const int t = opaque_int(tid);
#pragma unroll
    for (int k = 0; k < KPT; ++k)
      if (k < nrow && k * NT + t != victim) keep |= 1ull << k;
  } else if (need > 0) {
    uint32_t smask;
    const uint32_t sprefix = radix_score_regs<NT, KPT>(need, fk, win, nrow, ws, &smask);
    // candidates strictly above the threshold class, and the size of that class
    int above = 0, tied = 0;
#pragma unroll
    for (int k = 0; k < KPT; ++k)
      if (k < nrow && !((win >> k) & 1)) {
        above += (fk[k] & smask) > sprefix ? 1 : 0;
        tied += (fk[k] & smask) == sprefix ? 1 : 0;
      }
    // (work-group totals: taken as scalars, so the branches below stay uniform)
    above = __builtin_amdgcn_readfirstlane(block_reduce<NT>(above, sc.red_i, [](int a, int b) { return a + b; }));
    tied = __builtin_amdgcn_readfirstlane(block_reduce<NT>(tied, sc.red_i, [](int a, int b) { return a + b; }));
    const int take = need - above;  // from the threshold class
    uint32_t tprefix = 0, tmask = 0;
    const bool split_ties = take < tied;  // only when scores tie exactly at the threshold
    if (split_ties) {
      if (smask != 0xFFFFFFFFu) {  // the class is one exact score once fully resolved
        fail(SE_DEVERR_BAD_POSITIONS);
        return;
      }
      if (tied <= kWave) {
        // A small class (SnapKV's max pooling makes runs of up to kappa equal
        // scores, so its threshold class is nearly always one): its positions go
        // to LDS (the holes list is not written yet) and one wavefront finds the
        // take-th smallest, instead of radix passes over every slot's position
        // and score in memory.  Same kept set: the take lowest positions.
        int* const tpos = sc.holes;
        if (tid == 0) {
          sc.bcast[0] = 0;  // entries
          sc.bcast[2] = 0;  // found
        }
        __syncthreads();
        {
          uint64_t tm = 0;  // this thread's rows in the class
#pragma unroll
          for (int k = 0; k < KPT; ++k)
            if (k < nrow && !((win >> k) & 1) && fk[k] == sprefix) tm |= 1ull << k;
          const int t = opaque_int(tid);
          while (tm != 0) {  // a few rows in the whole work-group
            const int k = __builtin_ctzll(tm);
            tm &= tm - 1;
            const int i = atomicAdd(&sc.bcast[0], 1);
            tpos[i] = p.pos_pool[addr(k * NT + t)];
          }
        }
        __syncthreads();
        if (wave == 0) {
          const int v = lane < tied ? tpos[lane] : INT_MAX;
          int rank = 0;  // tied entries with a smaller position
          for (int j = 0; j < tied; ++j) rank += __shfl(v, j, kWave) < v ? 1 : 0;
          if (lane < tied && rank == take - 1) {
            sc.bcast[1] = v;
            sc.bcast[2] = 1;
          }
        }
        __syncthreads();
        if (sc.bcast[2] == 0) {  // no unique take-th position: repeated positions
          fail(SE_DEVERR_BAD_POSITIONS);
          return;
        }
        tprefix = 0xFFFFFFFFu - pos_key(sc.bcast[1]);  // keep iff pos <= the take-th smallest
        tmask = 0xFFFFFFFFu;
      } else {
        radix_top_slots<NT, uint32_t>(
            p, L, take, [](int32_t q, float) { return 0xFFFFFFFFu - pos_key(q); },
            [&](int32_t q, float u) { return (w == 0 || pos_key(q) < wthr) && float_key(u) == sprefix; }, sc,
            &tprefix, &tmask);
      }
    }
    const int t = opaque_int(tid);
#pragma unroll
    for (int k = 0; k < KPT; ++k)
      if (k < nrow && !((win >> k) & 1)) {
        const uint32_t m = fk[k] & smask;
        bool kp = m > sprefix;
        if (m == sprefix) {
          kp = true;
          if (split_ties)
            kp = ((0xFFFFFFFFu - pos_key(p.pos_pool[addr(k * NT + t)])) & tmask) >= tprefix;
        }
        if (kp) keep |= 1ull << k;
      }
  }

  // ---- the retained set must hold exactly B slots (distinct positions)
  {
    const int kept = block_reduce<NT>((int)__popcll(keep), sc.red_i, [](int a, int b) { return a + b; });
    if (kept != B) {
      fail(SE_DEVERR_BAD_POSITIONS);
      return;
    }
  }

  // ---- ranking: holes are evicted slots below B, movers kept slots at or above
  // B, both in slot order (row k, then wavefront, then lane)
  {
    const int t = opaque_int(tid);
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const int s = k * NT + t;
      const bool kp = (keep >> k) & 1;
      const uint64_t hb = __ballot(k < nrow && s < B && !kp);
      const uint64_t mb = __ballot(s >= B && kp);
      if (lane == 0) {
        ws.cnt_h[k * NW + wave] = __popcll(hb);
        ws.cnt_m[k * NW + wave] = __popcll(mb);
      }
    }
  }
  __syncthreads();
  int n_moves;
  {
    const int vh = tid < KPT * NW ? ws.cnt_h[tid] : 0;
    const int vm = tid < KPT * NW ? ws.cnt_m[tid] : 0;
    int th, tm;
    const int eh = block_exclusive_scan<NT>(vh, sc.scan, &th);
    const int em = block_exclusive_scan<NT>(vm, sc.scan, &tm);
    if (tid < KPT * NW) {
      ws.cnt_h[tid] = eh;
      ws.cnt_m[tid] = em;
    }
    n_moves = tm;
    if (th != tm) {  // cannot happen when exactly B slots are kept
      fail(SE_DEVERR_BAD_POSITIONS);
      return;
    }
  }
  __syncthreads();
  {
    const int t = opaque_int(tid);
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const int s = k * NT + t;
      const bool h = k < nrow && s < B && !((keep >> k) & 1);
      const uint64_t hb = __ballot(h);
      if (h) sc.holes[ws.cnt_h[k * NW + wave] + lane_prefix(hb)] = s;
    }
  }
  __syncthreads();
  {
    const int t = opaque_int(tid);
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const int s = k * NT + t;
      const bool m = s >= B && ((keep >> k) & 1);
      const uint64_t mb = __ballot(m);
      if (m) ws.movers[ws.cnt_m[k * NW + wave] + lane_prefix(mb)] = s;
    }
  }
  __syncthreads();

  if (p.moves != nullptr) {  // the moves are left to evict_move_kernel
    for (int r = tid; r < n_moves; r += NT) {
      p.moves[kMoveHoles + r] = sc.holes[r];
      p.moves[kMoveMovers + r] = ws.movers[r];
    }
    if (tid == 0) p.moves[0] = n_moves;
  } else {
  // ---- mover r's key and value rows go to hole r; one 16-byte chunk per
  // thread, and the threads of chunks 0 and 1 also carry the position and the
  // score (nothing else reads a mover's source entry or a hole's old one)
    constexpr int C = D / 8;            // chunks per row
    constexpr int TPM = 2 * C;          // threads per mover (key row, then value row)
    constexpr int MPP = NT / TPM;       // movers per pass
    const int c = tid % TPM;
    const int off = (c < C ? 0 : kPage * D) + (c % C) * 8;  // in bf16 elements
    int32_t* const side = c == 0 ? p.pos_pool : reinterpret_cast<int32_t*>(p.score_pool);
    auto row = [&](int s) -> uint4* {
      return reinterpret_cast<uint4*>(p.kv + (size_t)ws.bt[s >> 4] * 2 * kPage * D + (s & (kPage - 1)) * D + off);
    };
    int r = tid / TPM;
    for (; r + 3 * MPP < n_moves; r += 4 * MPP) {  // four movers in flight per thread
      const int s0 = ws.movers[r], s1 = ws.movers[r + MPP], s2 = ws.movers[r + 2 * MPP], s3 = ws.movers[r + 3 * MPP];
      const uint4 v0 = *row(s0), v1 = *row(s1), v2 = *row(s2), v3 = *row(s3);
      int32_t x0 = 0, x1 = 0, x2 = 0, x3 = 0;
      if (c < 2) {
        x0 = side[addr(s0)];
        x1 = side[addr(s1)];
        x2 = side[addr(s2)];
        x3 = side[addr(s3)];
      }
      const int d0 = sc.holes[r], d1 = sc.holes[r + MPP], d2 = sc.holes[r + 2 * MPP], d3 = sc.holes[r + 3 * MPP];
      *row(d0) = v0;
      *row(d1) = v1;
      *row(d2) = v2;
      *row(d3) = v3;
      if (c < 2) {
        side[addr(d0)] = x0;
        side[addr(d1)] = x1;
        side[addr(d2)] = x2;
        side[addr(d3)] = x3;
      }
    }
    for (; r < n_moves; r += MPP) {
      const int s0 = ws.movers[r], d0 = sc.holes[r];
      const uint4 v0 = *row(s0);
      int32_t x0 = 0;
      if (c < 2) x0 = side[addr(s0)];
      *row(d0) = v0;
      if (c < 2) side[addr(d0)] = x0;
    }
  }

  // ---- release: pages ceil(B/16) .. ceil(L/16)-1 hold nothing now
  const int f0 = ceil_div_dev(B, kPage);
  const int nf = n_pages - f0;
  if (p.freed_pages != nullptr)
    for (int i = tid; i < nf; i += NT) p.freed_pages[(size_t)unit * p.freed_stride + i] = ws.bt[f0 + i];
  if (tid == 0) {
    if (p.freed_count != nullptr) p.freed_count[unit] = nf;
    p.lengths[unit] = B;
  }
}

}  // namespace se
