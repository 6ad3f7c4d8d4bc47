// se_decode_attend: append the decode token, split-K paged GQA decode attention
// over a per-unit view, and the fused H2O score update.
//
// Math (Appendix A.1, eq. background-selected-attention; Appendix A.3, eq.
// background-h2o-score): for each query row a of a unit, z_j = scale * <q_a, k_j>
// over the read set, out_a = sum_j softmax(z)_j v_j, and with accumulation every
// read slot's score grows by its weight summed over the unit's G rows.
//
// Work decomposition.  A unit's visited pages are cut into n_split ranges (one
// range when there are enough units to fill the chip); one 512-thread
// work-group (eight wavefronts) streams one range, each wavefront one page at
// a time:
//   * QK layout: 8 lanes share a K row, each with D/8 columns (16-byte loads),
//     two passes cover the page's 16 rows; bf16 pair dot products with the G
//     query rows (v_dot2c_f32_bf16) and a 3-step DPP reduction give every lane
//     the G logits of its rows; each lane keeps one (row, head) pair.
//   * Pipeline: the physical pages of a wavefront's next 64 pages are fetched
//     by one vector load, and the next page's K and V are loaded while the
//     current page computes (two register buffers).
//   * Softmax: each wavefront keeps one reference maximum per head, raised
//     (and the running sums rescaled) only when a logit exceeds it by more than
//     2^8, so most pages need one exp2 per (row, head) and no cross-lane max.
//   * PV layout: lane owns two adjacent columns of the V block for all 16 rows
//     (one coalesced 256-byte row per load instruction across the wave); the
//     page's 16*G weights are broadcast through LDS.
// With one work-group per unit that work-group finishes the unit itself.  With
// several, each writes its partial (m, l, o) to the workspace and a second,
// one-work-group-per-unit kernel combines them in a fixed order, writes out and
// lse, runs the score epilogue and publishes the new length.  The kernel
// boundary orders the two passes across XCDs (each XCD has its own L2), which
// avoids a device-scope release/acquire (an L2 writeback and invalidate) in
// every work-group.
#include <mutex>
#include <type_traits>

#include "evict_core.h"
#include "quest_core.h"

namespace se {

struct AttendParams {
  const uint16_t* kv;
  int32_t* pos_pool;
  float* score_pool;
  uint16_t* meta_pool;
  const int32_t* block_table;
  int32_t* lengths;
  int64_t num_pages;
  int32_t hkv;
  int32_t max_pages;
  const uint16_t* q;
  const uint16_t* k_new;
  const uint16_t* v_new;
  const int32_t* new_pos;
  const int32_t* sel;
  int32_t top_k;
  // se_decode_step_quest: the kernel selects the pages itself (Quest bound +
  // top-k over the unit's candidate pages; candidates plus top_k must not
  // exceed kSelectMaxPages), attends over the selection and writes it to sel
  int32_t select;
  const uint16_t* meta;
  float scale;
  float scale_log2;
  int32_t max_len;
  int32_t n_visit_max;
  int32_t pps;
  int32_t n_split;
  int32_t accumulate;
  float* out;
  float* lse;
  float* logits;
  int32_t logits_stride;
  float* part;
  float* pbuf;
  float* mref;
  const int32_t* order;  // unit of each work-group slot (longest first), or null: identity
  int32_t* dev_err;
  // fused steady-state H2O eviction (se_decode_step_h2o)
  int32_t evict;
  int32_t budget;
  int32_t recent;
  int32_t* freed_pages;
  int32_t freed_stride;
  int32_t* freed_count;
};

struct AttendWs {
  size_t part, pbuf, mref, order, total;
};

inline AttendWs attend_ws_layout(int units, const SplitShape& s, int G, int D) {
  AttendWs w;
  size_t off = 0;
  w.part = off;
  off = align_up(off + (size_t)units * s.n_split * G * (D + 2) * 4, 256);
  w.pbuf = off;
  off = align_up(off + (size_t)units * s.n_visit * kPage * G * 4, 256);
  w.mref = off;
  off = align_up(off + (size_t)units * s.n_visit * G * 4, 256);
  w.order = off;
  off = align_up(off + (size_t)units * 4, 256);
  w.total = off;
  return w;
}

// Per-unit quantities both kernels derive the same way from the inputs.
struct UnitGeom {
  int unit, req, kvh, L, Lp, cur_page, n_visit;
  bool append, quest, bad;
};

__device__ __forceinline__ UnitGeom unit_geom(const AttendParams& p, int unit) {
  UnitGeom g;
  g.unit = unit;
  g.req = unit / p.hkv;
  g.kvh = unit - g.req * p.hkv;
  g.L = p.lengths[unit];
  g.append = p.k_new != nullptr;
  g.Lp = g.L + (g.append ? 1 : 0);
  g.quest = p.sel != nullptr;
  g.bad = g.L < 0 || g.Lp < 1 || g.Lp > p.max_len || g.Lp > p.max_pages * kPage;
  g.cur_page = g.bad ? 0 : (g.Lp - 1) / kPage;
  g.n_visit = g.bad ? 0 : (g.quest ? p.top_k + 1 : g.cur_page + 1);
  return g;
}

// After the unit's final (m, 1/l) per head are in fin_m / fin_il: the fused
// score update over every visited slot (eq. background-h2o-score, summed over
// the group; the new token's score is its weight) and the new length.
template <int G>
__device__ __forceinline__ float slot_weight(const AttendParams& p, size_t ubase_p, int vp, int rr,
                                             const float* fin_m, const float* fin_il) {
  float a = 0.f;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float w = p.pbuf[((ubase_p + vp) * kPage + rr) * G + h];
    const float mr = p.mref[(ubase_p + vp) * G + h];
    a += w * fast_exp2(mr - fin_m[h]) * fin_il[h];
  }
  return a;
}

// When one work-group holds a whole unit, the per-slot weights (fp16: each
// is rounded by at most 2^-11 relative before the fp32 score update) and the
// per-page reference maxima (fp32) of its first kWeightPages<G> visit pages
// stay in LDS instead of going through the workspace, which would add an HBM
// write and read of 16 B per slot to the step; the buffer is the eviction
// scratch's holes array, which only the general eviction uses, after the
// scores are written.
constexpr int kWeightCap = 9216;  // 32-bit words (>= kMaxBudget ints for the holes)
constexpr int kSelectMaxPages = kWeightCap / 2;  // fused Quest selection: block-table row + selection, scores
constexpr int kWeightMrCap = 2 * kWeightCap / kPage;  // reference maxima: one per (visit page, head)
template <int G, typename W>
constexpr int kWeightPages =
    (kWeightCap * 4 / (int)sizeof(W) / (kPage * G)) < 1024 ? kWeightCap * 4 / (int)sizeof(W) / (kPage * G) : 1024;
static_assert(kWeightCap >= kMaxBudget, "the weight buffer doubles as the holes array");
static_assert(kWeightPages<8, _Float16> * 8 <= kWeightMrCap && kWeightPages<4, _Float16> * 4 <= kWeightMrCap &&
                  kWeightPages<1, _Float16> <= kWeightMrCap,
              "reference maxima");
// The weight format of a kernel instantiation: fp32 where the units it takes
// fit the buffer that way (the 512-thread per-wavefront steady variant, at most
// wave_rows_pages pages, groups of up to 4), fp16 elsewhere (twice the pages).
template <int NT, bool kWaveRows, int G>
using WeightT = typename std::conditional<kWaveRows && NT == 512 && G <= 4, float, _Float16>::type;

// Where the score update finds the weights: visit pages below `cap` in the
// work-group's LDS buffer, the others in the workspace rows (global).
template <typename W>
struct WeightSrc {
  const W* lw;         // LDS [visit page][16][G]
  const float* lfac;  // LDS [visit page][G]: exp2(m_ref - m) / l, the page's factor per head
  const float* gw;   // workspace, same layout
  const float* gmr;
  int cap;
};

// A slot's weight summed over the group when its page's weights are in LDS.
template <int G, typename W>
__device__ __forceinline__ float slot_weight_lds(const WeightSrc<W>& src, int vp, int rr) {
  float a = 0.f;
#pragma unroll
  for (int h = 0; h < G; ++h) a += (float)src.lw[(vp * kPage + rr) * G + h] * src.lfac[vp * G + h];
  return a;
}

template <int G, typename W>
__device__ __forceinline__ float slot_weight_from(const WeightSrc<W>& src, int vp, int rr, const float* fin_m,
                                                  const float* fin_il) {
  float a = 0.f;
  if (vp < src.cap) {
    a = slot_weight_lds<G, W>(src, vp, rr);
  } else {
#pragma unroll
    for (int h = 0; h < G; ++h)
      a += src.gw[(vp * kPage + rr) * G + h] * fast_exp2(src.gmr[vp * G + h] - fin_m[h]) * fin_il[h];
  }
  return a;
}

__device__ __forceinline__ uint32_t pos_order(int32_t pos) { return (uint32_t)pos ^ 0x80000000u; }

// With se_decode_step_h2o, the step's eviction (eq. background-h2o-retention)
// is done here when it is the steady one-slot case: the unit is one slot over
// the budget and its recent window is the contiguous run of newest positions.
// Every slot's new score and position stay in registers; the victim is the
// non-window slot with the smallest (score, then larger position); the new
// token's slot (the last one) moves into it.  Anything else is left to the
// general eviction kernel that se_decode_step_h2o launches next.
// The general eviction of a unit in the epilogue (after its scores are written).
// The kernel calls it from one place, as an unlikely branch at the end of the
// epilogue, so that its code (a radix selection) sits after the hot path:
// instruction-cache misses cost a memory latency each in every work-group.
template <int NT, int D>
__device__ __forceinline__ void evict_in_epilogue(const AttendParams& p, const UnitGeom& g, const EvictScratch<NT>& sc) {
  __syncthreads();
  EvictJob job;
  job.kv = const_cast<uint16_t*>(p.kv);
  job.pos_pool = p.pos_pool;
  job.score_pool = p.score_pool;
  job.bt = p.block_table + (size_t)g.unit * p.max_pages;
  job.lengths = p.lengths;
  job.num_pages = p.num_pages;
  job.unit = g.unit;
  job.L = g.Lp;
  job.budget = p.budget;
  job.recent = p.recent;
  job.max_len = p.max_len;
  job.max_pages = p.max_pages;
  job.freed_pages = p.freed_pages;
  job.freed_stride = p.freed_stride;
  job.freed_count = p.freed_count;
  job.dev_err = p.dev_err;
  evict_unit<NT, D>(job, sc);
}

// The fused steady eviction (one slot over the budget, contiguous window) of a
// unit that one work-group streamed whole: every wavefront handles the slots of
// the pages it streamed (lane l: row l % 16 of its pages l / 16 + 4 j), whose
// positions and old scores it fetched as soon as its own stream ended (spos,
// su), so only LDS reads and arithmetic remain here before the reductions.
// The staged table is the unit's page table (staged index = logical page).
constexpr int kSteadyRows = 5;  // pages per wavefront up to 4 * kSteadyRows

// The steady eviction's one move: the newest slot (mover) into the victim's
// slot, with its key and value rows, position and score.  When the step
// appended, the newest slot's rows are the step's k_new / v_new, read from
// there rather than from the pool the append wrote, so nothing waits for the
// append's stores.
template <int D>
__device__ __forceinline__ void move_newest(const AttendParams& p, const UnitGeom& g, int pv, int victim, int pm,
                                            int mover, int32_t mpos, float mu) {
  if (victim == mover) return;
  const int tid = threadIdx.x;
  constexpr int R4 = D / 8;  // 16-byte chunks per row
  uint4* dst = reinterpret_cast<uint4*>(const_cast<uint16_t*>(p.kv) + (size_t)pv * (2 * kPage * D) + (victim & 15) * D);
  if (tid < 2 * R4) {
    const int part = tid / R4, c = tid - part * R4;  // part 0: key row, 1: value row
    const uint4* src;
    if (g.append && mover == g.L)
      src = reinterpret_cast<const uint4*>((part ? p.v_new : p.k_new) + ((size_t)g.req * p.hkv + g.kvh) * D);
    else
      src = reinterpret_cast<const uint4*>(p.kv + (size_t)pm * (2 * kPage * D) + (mover & 15) * D) + part * kPage * R4;
    dst[part * kPage * R4 + c] = src[c];
  }
  if (tid == 0) {
    p.pos_pool[(size_t)pv * kPage + (victim & 15)] = mpos;
    p.score_pool[(size_t)pv * kPage + (victim & 15)] = mu;
  }
}

// The steady epilogue's one barrier round: the work-group's count of window
// slots (sum) and its least eviction key with the slot holding it (equal keys,
// which only repeated positions give, resolve to the lower slot, so every thread
// agrees).  A thread without a candidate passes key ~0 and slot INT_MAX.  The
// scratch is free again only after the caller's next barrier.
template <int NT>
__device__ __forceinline__ void steady_fold(int& cnt, unsigned long long& key, int& slot, const EvictScratch<NT>& sc) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  auto take = [&](int c2, unsigned long long k2, int s2) {
    cnt += c2;
    if (k2 < key || (k2 == key && s2 < slot)) {
      key = k2;
      slot = s2;
    }
  };
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) take(__shfl_xor(cnt, o, kWave), __shfl_xor(key, o, kWave), __shfl_xor(slot, o, kWave));
  if (lane == 0) {
    sc.red_i[wave] = cnt;
    sc.red_u64[wave] = key;
    sc.scan[wave] = slot;
  }
  __syncthreads();
  cnt = 0;
  key = ~0ull;
  slot = INT_MAX;
#pragma unroll
  for (int w = 0; w < NT / kWave; ++w) take(sc.red_i[w], sc.red_u64[w], sc.scan[w]);
}

// The lower bound of the recent window, lo: when exactly w resident positions
// lie above lo, they are the w largest and every other slot is a candidate.
// With an append, the new position (the largest in order) gives lo at once;
// otherwise the largest resident position does, by one more reduction.
template <int NT>
__device__ __forceinline__ int64_t steady_window_lo(const AttendParams& p, const UnitGeom& g, int32_t pmax, int w,
                                                    int* red_i) {
  if (g.append) return (int64_t)p.new_pos[g.req] - w;
  pmax = block_reduce<NT>(pmax, red_i, [](int x, int y) { return x > y ? x : y; });
  return (int64_t)pmax - w;
}

template <int NT, int G, int D, typename W>
__device__ __forceinline__ bool finish_steady(const AttendParams& p, const UnitGeom& g, const float* fin_m,
                                              const float* fin_il, const int* lds_phys, const int* lds_vp,
                                              const WeightSrc<W>& wsrc, int32_t (&pos)[kSteadyRows],
                                              float (&unew)[kSteadyRows], int rbeg, int wr, int n_my,
                                              const EvictScratch<NT>& sc) {
  constexpr int KW = kSteadyRows;
  __shared__ int bc_pos;  // the mover's position and score
  __shared__ float bc_u;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int r = lane & (kPage - 1);
  // slot of row j of this lane, or -1
  auto slot_of = [&](int j) -> int {
    const int i = (lane >> 4) + 4 * j;
    if (i >= n_my) return -1;
    const int s = (rbeg + wr + 4 * i) * kPage + r;
    return s < g.Lp ? s : -1;
  };
  // pos / unew hold the fetched positions and old scores; the scores become the
  // new ones.  They are stored only after the last barrier: a barrier waits
  // for the work-group's outstanding stores, which under a full memory system
  // take tens of microseconds.
  uint32_t live = 0;
#pragma unroll
  for (int j = 0; j < KW; ++j) {
    const int s = slot_of(j);
    if (s >= 0) {
      live |= 1u << j;
      const int gi = s >> 4;
      unew[j] += slot_weight_lds<G, W>(wsrc, lds_vp[gi], r);  // every page is in LDS here
    }
  }
  auto store_scores = [&](int skip) {
#pragma unroll
    for (int j = 0; j < KW; ++j) {
      const int s = slot_of(j);
      if (((live >> j) & 1) && s != skip) p.score_pool[(size_t)lds_phys[s >> 4] * kPage + r] = unew[j];
    }
  };
  const int w = min(p.recent, p.budget);
  int32_t pmax = INT32_MIN;
#pragma unroll
  for (int j = 0; j < KW; ++j)
    if ((live >> j) & 1) pmax = max(pmax, pos[j]);
  const int64_t lo = steady_window_lo<NT>(p, g, pmax, w, sc.red_i);
  const int mover = g.Lp - 1;
  int cnt = 0;
  unsigned long long best = ~0ull;
  int victim = INT_MAX;
#pragma unroll
  for (int j = 0; j < KW; ++j) {
    if (!((live >> j) & 1)) continue;
    const int s = slot_of(j);
    if ((int64_t)pos[j] > lo) {
      ++cnt;
    } else {
      const unsigned long long key = ((unsigned long long)float_key(unew[j]) << 32) |
                                     (unsigned long long)(0xFFFFFFFFu - pos_order(pos[j]));
      if (key < best) {
        best = key;
        victim = s;
      }
    }
    if (s == mover) {
      bc_pos = pos[j];
      bc_u = unew[j];
    }
  }
  steady_fold<NT>(cnt, best, victim, sc);
  if (cnt != w) {  // the general eviction runs from the updated scores
    __syncthreads();
    store_scores(-1);
    return true;
  }
  // every store after the last barrier: the scores (the victim's slot takes the
  // mover's), the mover's row, position and score in the victim's slot
  store_scores(victim);
  move_newest<D>(p, g, lds_phys[victim >> 4], victim, lds_phys[mover >> 4], mover, bc_pos, bc_u);
  if (tid == 0) {
    p.lengths[g.unit] = p.budget;
    const int f0 = (p.budget + kPage - 1) / kPage;
    const int nf = (g.Lp + kPage - 1) / kPage - f0;
    if (p.freed_pages != nullptr && nf > 0) p.freed_pages[(size_t)g.unit * p.freed_stride] = lds_phys[f0];
    if (p.freed_count != nullptr) p.freed_count[g.unit] = nf;
  }
  return false;
}

// The same for units too long for finish_steady's per-wavefront rows: thread
// t handles slots t + k * NT, loaded here (branch-free, in groups).  lds_bt:
// the unit's page table staged in LDS, in page order.
template <int NT, int G, int D, typename W>
__device__ __forceinline__ bool finish_steady_strided(const AttendParams& p, const UnitGeom& g, const float* fin_m,
                                              const float* fin_il, const int* lds_bt, const WeightSrc<W>& wsrc,
                                              const EvictScratch<NT>& sc) {
  constexpr int KMAX = kMaxBudget / NT;  // slots per thread kept in registers
  int* const red_i = sc.red_i;
  unsigned long long* const red_k = sc.red_u64;
  __shared__ int bc[2];
  __shared__ float bc_u;
  const int tid = threadIdx.x;
  const size_t ubase_p = (size_t)g.unit * p.n_visit_max;
  // Every row's position and old score is loaded first, all in flight together
  // (one memory latency for the epilogue; rows past the end re-read the last
  // slot, a bad page reads page 0 and is discarded), then the weights are added;
  // the stores come after every load.
  float unew[KMAX];
  int32_t pos[KMAX];
  uint32_t live = 0;  // rows k that hold a resident slot of a valid page
  int badp = 0;
  const int32_t pos_new = g.append ? p.new_pos[g.req] : 0;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int s = min(tid + k * NT, g.Lp - 1);
    const int ph = lds_bt[s >> 4];
    const bool ok = ph >= 0 && (int64_t)ph < p.num_pages;
    if (ok && tid + k * NT < g.Lp) live |= 1u << k;
    badp |= (tid + k * NT < g.Lp && !ok) ? 1 : 0;
    const size_t a_ = (size_t)(ok ? ph : 0) * kPage + (s & (kPage - 1));
    unew[k] = p.score_pool[a_];
    pos[k] = p.pos_pool[a_];
  }
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int s = tid + k * NT;
    const int sc_ = min(s, g.Lp - 1);
    const float a = slot_weight_from<G, W>(wsrc, sc_ >> 4, sc_ & (kPage - 1), fin_m, fin_il);
    const bool lv = (live >> k) & 1;
    const bool is_new = g.append && s == g.L;
    unew[k] = lv ? (is_new ? 0.f : unew[k]) + a : 0.f;
    pos[k] = lv ? (is_new ? pos_new : pos[k]) : INT32_MIN;
  }
  // the new scores are stored after the last barrier (a barrier waits for the
  // work-group's outstanding stores), except when the general path evicts
  auto store_scores = [&](int skip) {
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const int s = tid + k * NT;
      if (((live >> k) & 1) && s != skip) p.score_pool[(size_t)lds_bt[s >> 4] * kPage + (s & (kPage - 1))] = unew[k];
    }
  };
  badp = block_reduce<NT>(badp, red_i, [](int x, int y) { return x | y; });
  const int w = min(p.recent, p.budget);
  int32_t pmax = INT32_MIN;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) pmax = max(pmax, pos[k]);
  pmax = block_reduce<NT>(pmax, red_i, [](int x, int y) { return x > y ? x : y; });
  const int64_t lo = (int64_t)pmax - w;  // the window is the positions above lo when contiguous
  int cnt = 0;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) cnt += (tid + k * NT < g.Lp && (int64_t)pos[k] > lo) ? 1 : 0;
  cnt = block_reduce<NT>(cnt, red_i, [](int x, int y) { return x + y; });
  if (badp || cnt != w) {  // the general eviction runs from the updated scores
    store_scores(-1);
    return true;
  }
  unsigned long long best = ~0ull;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int s = tid + k * NT;
    if (s < g.Lp && (int64_t)pos[k] <= lo) {
      const unsigned long long key = ((unsigned long long)float_key(unew[k]) << 32) |
                                     (unsigned long long)(0xFFFFFFFFu - pos_order(pos[k]));
      best = key < best ? key : best;
    }
  }
  const unsigned long long kmin =
      block_reduce<NT>(best, red_k, [](unsigned long long x, unsigned long long y) { return x < y ? x : y; });
  const int mover = g.Lp - 1;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    const int s = tid + k * NT;
    if (s < g.Lp && (int64_t)pos[k] <= lo) {
      const unsigned long long key = ((unsigned long long)float_key(unew[k]) << 32) |
                                     (unsigned long long)(0xFFFFFFFFu - pos_order(pos[k]));
      if (key == kmin) bc[0] = s;
    }
    if (s == mover) {
      bc[1] = pos[k];
      bc_u = unew[k];
    }
  }
  __syncthreads();
  const int victim = bc[0];
  store_scores(victim);
  move_newest<D>(p, g, lds_bt[victim >> 4], victim, lds_bt[mover >> 4], mover, bc[1], bc_u);
  if (tid == 0) {
    p.lengths[g.unit] = p.budget;
    const int f0 = (p.budget + kPage - 1) / kPage;
    const int nf = (g.Lp + kPage - 1) / kPage - f0;
    if (p.freed_pages != nullptr && nf > 0) p.freed_pages[(size_t)g.unit * p.freed_stride] = lds_bt[f0];
    if (p.freed_count != nullptr) p.freed_count[g.unit] = nf;
  }
  return false;
}


// The score update of every visited slot, BATCH slots per thread at a time with
// all of a batch's loads issued before its stores.
template <int NT, int G, typename W>
__device__ __forceinline__ void accumulate_unit(const AttendParams& p, const UnitGeom& g, const float* fin_m,
                                                const float* fin_il, const WeightSrc<W>& wsrc) {
  constexpr int BATCH = 8;
  const size_t ubase_p = (size_t)g.unit * p.n_visit_max;
  const int32_t* bt = p.block_table + (size_t)g.unit * p.max_pages;
  float fm[G], fil[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    fm[h] = fin_m[h];
    fil[h] = fin_il[h];
  }
  const int n = g.n_visit * kPage;
  for (int b0 = threadIdx.x; b0 < n; b0 += NT * BATCH) {
    int ph[BATCH];
    float a[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int idx = b0 + j * NT;
      const int vp = idx >> 4;
      const int rr = idx & (kPage - 1);
      int lp = vp;
      bool ok = idx < n;
      if (ok && g.quest) {
        lp = vp < p.top_k ? p.sel[(size_t)g.unit * p.top_k + vp] : g.cur_page;
        ok = lp >= 0 && (vp >= p.top_k || lp < g.cur_page);
      }
      ok = ok && lp * kPage + rr < g.Lp;
      ph[j] = ok ? bt[lp] : -1;
      a[j] = ok ? slot_weight_from<G, W>(wsrc, vp, rr, fm, fil) : 0.f;
    }
    float u[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int idx = b0 + j * NT;
      const int rr = idx & (kPage - 1);
      const bool ok = ph[j] >= 0 && (int64_t)ph[j] < p.num_pages;
      const int vp = idx >> 4;
      const bool fresh = g.append && !g.quest ? vp * kPage + rr == g.L
                                               : (g.append && vp >= p.top_k && g.cur_page * kPage + rr == g.L);
      u[j] = ok && !fresh ? p.score_pool[(size_t)ph[j] * kPage + rr] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int rr = (b0 + j * NT) & (kPage - 1);
      if (ph[j] >= 0 && (int64_t)ph[j] < p.num_pages) p.score_pool[(size_t)ph[j] * kPage + rr] = u[j] + a[j];
    }
  }
}

// The score update and, with se_decode_step_h2o, the general eviction of a
// unit, after its final (m, 1/l) per head are in fin_m / fin_il.  The weights
// of visit pages below wcap come from the work-group's LDS buffer (lds_w,
// lds_mr), the others from the workspace.
// Returns true when the unit still needs the general eviction (which then sets
// its length and freed pages).
template <int NT, int G, bool kCanEvict, typename W>
__device__ __forceinline__ bool finish_unit(const AttendParams& p, const UnitGeom& g, const float* fin_m,
                                            const float* fin_il, const W* lds_w, const float* lds_mr, int wcap) {
  const int tid = threadIdx.x;
  const size_t ubase_p = (size_t)g.unit * p.n_visit_max;
  const WeightSrc<W> wsrc{lds_w, lds_mr, p.pbuf + ubase_p * kPage * G, p.mref + ubase_p * G, wcap};
  if (p.accumulate) accumulate_unit<NT, G, W>(p, g, fin_m, fin_il, wsrc);
  if constexpr (kCanEvict) {
    if (p.evict && !g.quest && g.Lp > p.budget) return true;
  }
  if (tid == 0) {
    if (g.append) p.lengths[g.unit] = g.Lp;
    if (kCanEvict && p.evict && p.freed_count != nullptr) p.freed_count[g.unit] = 0;
  }
  return false;
}

// Per-page coordinates a wavefront needs before it loads the page.
constexpr int kMaxGroupPages = 1024;  // pages one work-group streams at most
// Work-group sizes: 512 threads (eight wavefronts, two work-groups per compute
// unit, the default) or 1024 (sixteen, one per compute unit) when the launch
// has at most one work-group per compute unit anyway: a unit then needs no
// split (and no combine pass).
constexpr int kAttendThreads = 512;
constexpr int kAttendThreadsWide = 1024;

// Share of a work-group's pages per wavefront slot rank, in percent.  Wavefront
// w runs on SIMD w % 4 in slot w / 4; with equal shares a slot's wavefronts end
// after those of the slots before it (memory requests of older wavefronts are
// served first: ~15 % later for the second slot), so earlier slots take more
// pages.  A page's wavefront depends only on its index: the results do not
// depend on timing.
template <int NR>
struct RankWeights;
template <>
struct RankWeights<2> {
  static constexpr int w[2] = {58, 42};
};
template <>
struct RankWeights<4> {
  static constexpr int w[4] = {34, 26, 21, 19};
};

struct PageRef {
  int vp;      // index in the unit's visit order (workspace row)
  int lp;      // logical page
  int phys;    // physical page, or -1 when the page is skipped
  int nrows;   // resident rows of the page
  int rn;      // row of the appended token in this page, or -1
  bool tail;   // a prefetch past the wavefront's last page (its loads are not used)
};

// (row, head) pairs a lane keeps per page: heads own_head + 4k, k < kPairs.
// Groups of 8 take two passes of the 4-head reduction over the same K
// registers.
template <int G>
constexpr int kPairs = G > 4 ? G / 4 : 1;
template <int G>
constexpr int kPassHeads = G < 4 ? G : 4;  // heads per pass

// Lane coordinates of the two layouts (see the kernel).
template <int D>
struct Lanes {
  static constexpr int QC = D / 8;        // K columns per lane (QK layout: 8 lanes per row)
  static constexpr int QW = QC / 2;       // bf16 pairs per lane per head
  static constexpr int K4 = QC / 8;       // 16-byte loads per lane per K row
  static constexpr int RS = 128 / D;      // row sets of the PV layout
  static constexpr int RPL = kPage / RS;  // rows per lane (PV layout)
  static constexpr int HP = D / 2;        // lanes per row set (two columns each)
  int r8, j8, own_row, own_head, col, rs;
  bool owns;
  uint32_t koff;  // bytes from a page's start to the lane's K piece of row r8
  uint32_t voff;  // bytes from a page's V block to the lane's column pair of row rs * RPL
};

// Loads of one page: K rows r8 and r8+8 (QK layout) and the V column pair
// (PV layout) of every row the lane owns.  The page base is wave-uniform
// (scalar registers) and each row is a constant offset from the lane's offset,
// so no load needs per-lane address arithmetic.  Rows past the page's resident
// rows are read too (they lie inside the page): their logits are masked and
// their value columns cleared before the PV update (pv_page).  A tail
// prefetch (past the wavefront's last page) reads the last page again with
// every lane at the page's first bytes: a few cache lines instead of the
// page, which the streaming loads have already let go from the L2.
// K/V page data is read once per step: nontemporal loads (streaming cache
// policy), so the stream does not push the block tables, positions, scores and
// the kernel's code out of the L2.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 stream_load16(const char* ptr) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(ptr));
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <int D>
__device__ __forceinline__ const char* page_base(const AttendParams& p, const PageRef& pr) {
  return reinterpret_cast<const char*>(p.kv) + (size_t)pr.phys * (2 * kPage * D * 2);
}

template <int D>
__device__ __forceinline__ void load_k(const AttendParams& p, const Lanes<D>& ln, const PageRef& pr,
                                       uint4 (&kb)[2 * Lanes<D>::K4]) {
  constexpr int K4 = Lanes<D>::K4;
  const char* kpage = page_base<D>(p, pr) + (pr.tail ? 0u : ln.koff);
#pragma unroll
  for (int pass = 0; pass < 2; ++pass)
#pragma unroll
    for (int i = 0; i < K4; ++i)
      kb[pass * K4 + i] = stream_load16(kpage + pass * 8 * D * 2 + i * 16);
}

template <int D>
__device__ __forceinline__ void load_v(const AttendParams& p, const Lanes<D>& ln, const PageRef& pr,
                                       uint32_t (&vb)[Lanes<D>::RPL]) {
  constexpr int RPL = Lanes<D>::RPL;
  const char* vpage = page_base<D>(p, pr) + kPage * D * 2 + (pr.tail ? 0u : ln.voff);
#pragma unroll
  for (int i = 0; i < RPL; ++i) vb[i] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(vpage + i * D * 2));
}

// Reduce-scatter of the 8 lanes that share two K rows: on entry a[h] / b[h]
// are the lane's partial dot products of rows r8 / r8+8 with head h; on exit
// lane j8 holds the full sum for row r8 + 8*bit2(j8) and head j8 & 3.  Each
// step halves the values a lane keeps and adds its partner's copy of them
// (partners j8^7, j8^2, j8^1 via DPP row_half_mirror and quad permutations),
// so no lane ever selects by a computed index.
template <int G>
__device__ __forceinline__ float row_reduce_scatter(const float (&a)[G], const float (&b)[G], int j8) {
  constexpr int kDppHalfMirror = 0x141;
  const bool b2 = (j8 & 4) != 0, b1 = (j8 & 2) != 0, b0 = (j8 & 1) != 0;
  float k[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float keep = b2 ? b[h] : a[h];
    const float send = b2 ? a[h] : b[h];
    k[h] = keep + dpp_f<kDppHalfMirror>(send);
  }
  if constexpr (G == 4) {
    const float k0 = b1 ? k[2] : k[0], s0 = b1 ? k[0] : k[2];
    const float k1 = b1 ? k[3] : k[1], s1 = b1 ? k[1] : k[3];
    const float t0 = k0 + dpp_f<kQuadXor2>(s0);
    const float t1 = k1 + dpp_f<kQuadXor2>(s1);
    const float kk = b0 ? t1 : t0, ss = b0 ? t0 : t1;
    return kk + dpp_f<kQuadXor1>(ss);
  } else if constexpr (G == 2) {
    const float t0 = k[0] + dpp_f<kQuadXor2>(k[0]);
    const float t1 = k[1] + dpp_f<kQuadXor2>(k[1]);
    const float kk = b0 ? t1 : t0, ss = b0 ? t0 : t1;
    return kk + dpp_f<kQuadXor1>(ss);
  } else {
    static_assert(G == 1, "passes of 1, 2 or 4 query heads");
    const float t = k[0] + dpp_f<kQuadXor2>(k[0]);
    return t + dpp_f<kQuadXor1>(t);
  }
}

// Running per-wavefront softmax state: a reference maximum per head (log2
// units, uniform across the wavefront), the lane's share of the head's sum and
// of the weighted V columns it owns.
template <int G>
struct WaveSoftmax {
  float m_ref[G];
  float o_acc[G][2];
  float l_own[kPairs<G>];
  float m_own[kPairs<G>];  // m_ref of the lane's heads
};

// Logits of the lane's (row, head) pairs for one page, one pass of up to four
// heads at a time over the K registers.  The query rows are read from LDS (one
// copy per work-group) instead of being held in registers, which leaves room
// for a second page in flight.
template <int D, int G>
__device__ __forceinline__ void qk_page(const Lanes<D>& ln, const uint4 (&kb)[2 * Lanes<D>::K4],
                                        const uint32_t (*lds_q)[D / 2], float (&z)[kPairs<G>]) {
  constexpr int K4 = Lanes<D>::K4, QW = Lanes<D>::QW, GH = kPassHeads<G>;
#pragma unroll
  for (int k = 0; k < kPairs<G>; ++k) {
    float accA[GH], accB[GH];
#pragma unroll
    for (int h = 0; h < GH; ++h) {
      accA[h] = 0.f;
      accB[h] = 0.f;
    }
#pragma unroll
    for (int i = 0; i < K4; ++i) {
      const uint32_t ka[4] = {kb[i].x, kb[i].y, kb[i].z, kb[i].w};
      const uint32_t kc[4] = {kb[K4 + i].x, kb[K4 + i].y, kb[K4 + i].z, kb[K4 + i].w};
#pragma unroll
      for (int h = 0; h < GH; ++h) {
        const uint4 qv = reinterpret_cast<const uint4*>(&lds_q[4 * k + h][ln.j8 * QW])[i];
        const uint32_t qw[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          accA[h] = dot2bf16(qw[e], ka[e], accA[h]);
          accB[h] = dot2bf16(qw[e], kc[e], accB[h]);
        }
      }
    }
    z[k] = row_reduce_scatter<GH>(accA, accB, ln.j8);
  }
}

// Reference update, weight of the lane's pair, its workspace copy, and the
// weights' broadcast through LDS (the page's PV follows).
template <int D, int G, typename W>
__device__ __forceinline__ void softmax_page(const AttendParams& p, const Lanes<D>& ln,
                                             const PageRef& pr, const float (&z)[kPairs<G>], WaveSoftmax<G>& ws,
                                             float* lds_pw, int lane, int unit, size_t ubase_p,
                                             W* lds_w, float* lds_mr, int wcap) {
  constexpr int NP = kPairs<G>, GH = kPassHeads<G>;
  constexpr float kBump = 8.0f;  // rescale only when a logit beats the reference by 2^8
  const bool valid = ln.owns && ln.own_row < pr.nrows;
  float z2[NP];
  bool need = false;
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    z2[k] = valid ? z[k] * p.scale_log2 : -INFINITY;
    if (p.logits != nullptr && valid)
      p.logits[((size_t)unit * G + ln.own_head + 4 * k) * p.logits_stride + pr.lp * kPage + ln.own_row] =
          z[k] * p.scale;
    need = need || (valid && (z2[k] > ws.m_own[k] + kBump));
  }
  if (__ballot(need) != 0) {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      float mx = z2[k];  // lanes of one head differ in lane bits 2..5
      mx = fmaxf(mx, shfl_xor_f(mx, 4));
      mx = fmaxf(mx, shfl_xor_f(mx, 8));
      mx = fmaxf(mx, shfl_xor_f(mx, 16));
      mx = fmaxf(mx, shfl_xor_f(mx, 32));
      // lane h (< GH) is row 0 of head 4k + h, so it holds that head's page maximum
#pragma unroll
      for (int h = 0; h < GH; ++h) {
        const int hh = 4 * k + h;
        const float mh = fmaxf(ws.m_ref[hh], __shfl(mx, h, kWave));
        const float f = fast_exp2(ws.m_ref[hh] - mh);
        ws.o_acc[hh][0] *= f;
        ws.o_acc[hh][1] *= f;
        ws.m_ref[hh] = mh;
      }
      const float m_new = fmaxf(ws.m_own[k], mx);
      ws.l_own[k] *= fast_exp2(ws.m_own[k] - m_new);
      ws.m_own[k] = m_new;
    }
  }
  float pj[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    pj[k] = valid ? fast_exp2(z2[k] - ws.m_own[k]) : 0.f;
    ws.l_own[k] += pj[k];
  }
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int hh = ln.own_head + 4 * k;
    if (pr.vp < wcap) {
      if (ln.owns) lds_w[(pr.vp * kPage + ln.own_row) * G + hh] = (W)pj[k];
      if (lane < GH) lds_mr[pr.vp * G + lane + 4 * k] = ws.m_own[k];
    } else if (p.accumulate) {
      if (ln.owns) p.pbuf[((ubase_p + pr.vp) * kPage + ln.own_row) * G + hh] = pj[k];
      if (lane < GH) p.mref[(ubase_p + pr.vp) * G + lane + 4 * k] = ws.m_own[k];
    }
    if (ln.owns) lds_pw[ln.own_row * G + hh] = pj[k];
  }
  wave_lds_sync();
}

// o += P V for one page, the weights read back from LDS.
template <int D, int G>
__device__ __forceinline__ void pv_page(const Lanes<D>& ln, const uint32_t (&vb)[Lanes<D>::RPL], int nrows,
                                        WaveSoftmax<G>& ws, const float* lds_pw) {
  constexpr int RPL = Lanes<D>::RPL;
  // bf16 -> fp32 by byte permutes whose selectors are per row (scalar for
  // D = 128): rows past the resident ones become zeros, since a zero weight
  // times arbitrary bits (Inf, NaN) would not stay zero
  constexpr uint32_t kLo = 0x01000c0cu, kHi = 0x03020c0cu, kZero = 0x0c0c0c0cu;
#pragma unroll
  for (int i = 0; i < RPL; ++i) {
    const int rr = ln.rs * RPL + i;
    const bool ok = rr < nrows;
    const float v0 = __uint_as_float(__builtin_amdgcn_perm(0u, vb[i], ok ? kLo : kZero));
    const float v1 = __uint_as_float(__builtin_amdgcn_perm(0u, vb[i], ok ? kHi : kZero));
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ph = lds_pw[rr * G + h];
      ws.o_acc[h][0] = fmaf(ph, v0, ws.o_acc[h][0]);
      ws.o_acc[h][1] = fmaf(ph, v1, ws.o_acc[h][1]);
    }
  }
  wave_lds_sync();
}

// se_decode_step_quest's selection inside the attention kernel (one work-group
// per unit): the candidates' block-table row, the selection after it and the
// page scores live in the weight buffer, unused by Quest.  The selection goes
// to sel at the end of the kernel (a store before a barrier would hold the
// barrier until it completes).  Returns the selection in LDS.  When every
// candidate page is in the pool and there are at least top_k of them (and the
// current page is in the pool), the selection's output step also writes the
// staged page list (lds_phys / lds_lp / lds_vp: the selected pages in rank
// order, then the current page) and *n_staged is top_k + 1; else *n_staged is
// -1 and the kernel stages the pages from the selection, skipping bad ones.
template <int NT, int D, int G>
__device__ __forceinline__ const int* fused_quest_select(const AttendParams& p, int unit, int req, int kvh,
                                                         int n_cand, int cur_page, int ph_cur, float* lds_w,
                                                         int* lds_phys, int* lds_lp, int* lds_vp,
                                                         const EvictScratch<NT>& esc, int* n_staged) {
  __shared__ unsigned s_hist2[256];
  __shared__ int s_badc;
  const int tid = threadIdx.x;
  const int Hq = p.hkv * G;
  int* const sbt = reinterpret_cast<int*>(lds_w);
  int* const ssel = sbt + n_cand;  // n_cand + top_k <= kSelectMaxPages
  float* const ssc = lds_w + kSelectMaxPages;
  if (tid == 0) s_badc = 0;  // set below only after the next barrier
  int badc = 0;
  for (int i = tid; i < n_cand; i += NT) {
    int ph = p.block_table[(size_t)unit * p.max_pages + i];
    if (ph < 0 || (int64_t)ph >= p.num_pages) {
      badc = 1;
      ph = -1;
    }
    sbt[i] = ph;
  }
  if (badc) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
  if (tid < 256) {
    esc.hist[tid] = 0;
    s_hist2[tid] = 0;
  }
  __syncthreads();
  if (badc) s_badc = 1;
  unit_bounds<NT, D, G>(p.meta, p.q + ((size_t)req * Hq + (size_t)kvh * G) * D, p.scale, n_cand, sbt, ssc, nullptr,
                        esc.hist, s_hist2);
  __syncthreads();
  const int top_k = p.top_k;
  // (every candidate lies before the current page unless the step does not
  // append and the length ends a page; the staging loop checks that case)
  const bool direct = __builtin_amdgcn_readfirstlane((int)(s_badc == 0 && n_cand >= top_k && n_cand <= cur_page &&
                                                           p.n_split == 1 && top_k < kMaxGroupPages && ph_cur >= 0 &&
                                                           (int64_t)ph_cur < p.num_pages)) != 0;
  unit_topk<NT>(
      n_cand, top_k, ssc,
      [&](int r, int b) {
        ssel[r] = b;
        if (direct) {  // b >= 0: n_cand >= top_k
          lds_phys[r] = sbt[b];
          lds_lp[r] = b;
          lds_vp[r] = r;
        }
      },
      esc.hist, s_hist2, esc.bcast, true);
  if (direct && tid == 0) {
    lds_phys[top_k] = ph_cur;
    lds_lp[top_k] = cur_page;
    lds_vp[top_k] = top_k;
  }
  __syncthreads();
  *n_staged = direct ? top_k + 1 : -1;
  return ssel;
}

// kWaveRows: the fused steady eviction keeps each wavefront's own slots
// (finish_steady; units of at most kWaveRowsPages pages), else thread-strided
// slots (finish_steady_strided).  Two instantiations, chosen on the host from
// the step's length bound, since carrying both paths costs the shorter one
// registers.
template <int D, int G, int NT, bool kWaveRows, bool kQuest>
__global__ __launch_bounds__(NT, 4) void decode_attend_kernel(const AttendParams p) {
  constexpr int NW = NT / kWave;  // wavefronts per work-group
  using LN = Lanes<D>;
  constexpr int QC = LN::QC, QW = LN::QW, K4 = LN::K4, RS = LN::RS, RPL = LN::RPL, HP = LN::HP;

  constexpr int NP = kPairs<G>, GH = kPassHeads<G>;
  // the wavefronts' partial outputs go through LDS up to four heads at a time
  // (groups of 8 take two rounds), which keeps the work-group's LDS within two
  // work-groups per compute unit
  constexpr int GO = GH, NRND = G / GO;
  __shared__ float lds_p[NW][kPage * G];
  __shared__ float lds_m[NW][G];
  __shared__ float lds_l[NW][G];
  __shared__ float lds_o[NW][GO][D];
  __shared__ float fin_m[G];
  __shared__ float fin_il[G];
  __shared__ int lds_phys[kMaxGroupPages];
  __shared__ int lds_lp[kMaxGroupPages];
  __shared__ int lds_vp[kMaxGroupPages];
  __shared__ uint32_t lds_q[G][D / 2];  // the unit's G query rows (bf16 pairs)
  __shared__ float lds_w[kWeightCap];    // per-slot weights, then the eviction's holes
  __shared__ float lds_mr[kWeightMrCap];
  using W = WeightT<NT, kWaveRows, G>;
  W* const lds_wh = reinterpret_cast<W*>(lds_w);
  SE_EVICT_SCRATCH_WITH_HOLES(NT, esc, reinterpret_cast<int*>(lds_w));
  __shared__ int lds_scan[NT / kWave + 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int uslot = blockIdx.x / p.n_split;
  const int unit = p.order != nullptr ? p.order[uslot] : uslot;
  const int split = blockIdx.x - uslot * p.n_split;
  const UnitGeom g = unit_geom(p, unit);
  const int req = g.req, kvh = g.kvh, L = g.L, Lp = g.Lp, cur_page = g.cur_page;
  const bool append = g.append, bad = g.bad;
  constexpr bool quest = kQuest;  // a selection is given (sel != nullptr) exactly in the kQuest instantiations
  const int Hq = p.hkv * G;
  const int vbeg = split * p.pps;
  const int vend = min(vbeg + p.pps, g.n_visit);
  const size_t ubase_p = (size_t)unit * p.n_visit_max;  // page-indexed workspace rows
  // the score update's weights of visit pages below wcap stay in LDS (this
  // work-group holds the whole unit); the rest go to the workspace.  The fused
  // Quest selection keeps its results in the same buffer (and never accumulates).
  const bool select = kQuest && p.select;
  const int wcap = (p.accumulate && p.n_split == 1 && !select) ? kWeightPages<G, W> : 0;

  // QK layout: lane = 8*r8 + j8 reads columns [j8*QC, (j8+1)*QC) of rows r8
  // (pass A) and r8 + 8 (pass B).  After the 8-lane reduction, lane j8 < 4
  // keeps head j8 of row r8 and lane j8 >= 4 head j8-4 of row r8+8: each lane
  // owns one (row, head) pair of the page per pass of four heads.  PV layout:
  // two adjacent columns, RPL rows.
  LN ln;
  ln.r8 = lane >> 3;
  ln.j8 = lane & 7;
  ln.own_row = ln.r8 + ((ln.j8 & 4) ? 8 : 0);
  ln.own_head = ln.j8 & 3;
  ln.owns = ln.own_head < G;
  ln.col = 2 * (lane % HP);
  ln.rs = lane / HP;
  ln.koff = (uint32_t)(ln.r8 * D + ln.j8 * QC) * 2u;
  ln.voff = (uint32_t)(ln.rs * RPL * D + ln.col) * 2u;
  const int j8 = ln.j8;
  const int col = ln.col;

  {
    const uint4* qsrc = reinterpret_cast<const uint4*>(p.q + ((size_t)req * Hq + (size_t)kvh * G) * D);
    if (tid < G * D / 8) reinterpret_cast<uint4*>(&lds_q[0][0])[tid] = qsrc[tid];
  }

  WaveSoftmax<G> ws;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    ws.m_ref[h] = -INFINITY;
    ws.o_acc[h][0] = 0.f;
    ws.o_acc[h][1] = 0.f;
  }
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    ws.l_own[k] = 0.f;
    ws.m_own[k] = -INFINITY;
  }

  const uint16_t* knew_row = append ? p.k_new + ((size_t)req * p.hkv + kvh) * D : nullptr;
  const uint16_t* vnew_row = append ? p.v_new + ((size_t)req * p.hkv + kvh) * D : nullptr;

  // ---- fused Quest selection (se_decode_step_quest; one work-group per unit).
  // The current page's physical id is fetched first: its load overlaps the
  // selection.
  const int n_cand = select && !bad ? L / kPage : 0;  // complete pages before the current one
  const int* lds_sel = nullptr;
  int ph_cur = -1;
  int n_staged = -1;  // >= 0: the selection staged the pages itself
  if constexpr (kQuest) {
    if (select) {
      if (!bad) ph_cur = p.block_table[(size_t)unit * p.max_pages + cur_page];
      lds_sel = fused_quest_select<NT, D, G>(p, unit, req, kvh, n_cand, cur_page, ph_cur, lds_w, lds_phys, lds_lp,
                                             lds_vp, esc, &n_staged);
    }
  }
  auto store_sel = [&]() {
    if constexpr (kQuest) {
      if (select)
        for (int i = tid; i < p.top_k; i += NT) const_cast<int32_t*>(p.sel)[(size_t)unit * p.top_k + i] = lds_sel[i];
    }
  };

  // ---- this work-group's pages: visit index, logical and physical ids of the
  // pages it must read, compacted and staged in LDS once, so the page stream
  // below never waits on a dependent table load or branches around a page
  const int n_range = n_staged >= 0 ? 0 : max(0, vend - vbeg);
  bool bad_sel = false, bad_page = false;
  int n_grp = n_staged >= 0 ? n_staged : 0;
  for (int i0 = 0; i0 < n_range; i0 += NT) {
    const int i = i0 + tid;
    const int vp = vbeg + i;
    int lp = vp;
    int ph = -1;
    if (i < n_range) {
      bool ok = true;
      if (quest) {
        lp = vp < p.top_k ? (select ? lds_sel[vp] : p.sel[(size_t)unit * p.top_k + vp]) : cur_page;
        if (lp < 0) ok = false;
        if (lp >= 0 && vp < p.top_k && lp >= cur_page) {
          bad_sel = true;
          ok = false;
        }
      }
      if (ok) {
        if (select)  // the selected pages' ids are in the staged block-table row
          ph = lp < n_cand ? reinterpret_cast<const int*>(lds_w)[lp] : ph_cur;
        else
          ph = p.block_table[(size_t)unit * p.max_pages + lp];
        if (ph < 0 || (int64_t)ph >= p.num_pages) {
          bad_page = true;
          ph = -1;
        }
      }
    }
    int total;
    const int rank = block_exclusive_scan<NT>(ph >= 0 ? 1 : 0, lds_scan, &total);
    if (ph >= 0) {
      lds_phys[n_grp + rank] = ph;
      lds_lp[n_grp + rank] = lp;
      lds_vp[n_grp + rank] = vp;
    }
    n_grp += total;
  }
  if (bad_sel) set_error(p.dev_err, SE_DEVERR_BAD_SELECTION);
  if (bad_page) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);

  if (n_staged < 0) __syncthreads();  // the staged tables (else the selection's last barrier)

  // Pages of this wavefront: the staged entries of its slot rank (a contiguous
  // share of the list, sized by kRankWeight), interleaved over the rank's four
  // wavefronts.
  constexpr int NR = NW / 4;  // slot ranks
  static_assert(NW % 4 == 0, "four SIMDs");
  const int srank = wave >> 2, wr = wave & 3;
  const int gl = n_grp - 1;  // the last staged entry
  int rbeg = 0, rcnt = 0, max_rcnt = 0, owner_rank = 0, owner_beg = 0;
  {
    int cum = 0, b = 0;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      cum += RankWeights<NR>::w[r];
      const int e = (n_grp * cum + 50) / 100;
      if (r == srank) {
        rbeg = b;
        rcnt = e - b;
      }
      if (gl >= b && gl < e) {
        owner_rank = r;
        owner_beg = b;
      }
      max_rcnt = max(max_rcnt, e - b);
      b = e;
    }
  }
  const int n_my = wr < rcnt ? (rcnt - wr + 3) / 4 : 0;

  // ---- append: the new token's page is the last one visited (the last staged
  // entry, when it is valid); the wavefront that streams it writes the row into
  // the pool before its first load and waits for its stores, so no other
  // wavefront waits for the append.  Nothing else reads that page in this pass
  // except the epilogue, which comes after a barrier.
  {
    const int new_vp = quest ? p.top_k : cur_page;
    const bool mine_new = append && !bad && new_vp >= vbeg && new_vp < vend && gl >= 0 && lds_vp[gl] == new_vp;
    const int owner_wr = (gl - owner_beg) & 3;
    if (mine_new && srank == owner_rank && wr == owner_wr) {
      const int ph = lds_phys[gl];
      const int rn = L - cur_page * kPage;
      uint16_t* kdst = const_cast<uint16_t*>(p.kv) + (size_t)ph * (2 * kPage * D) + rn * D;
      uint16_t* vdst = kdst + kPage * D;
      constexpr int R4 = D / 8;  // 16-byte chunks per row
      if (lane < 2 * R4) {
        const uint4* src = reinterpret_cast<const uint4*>(lane < R4 ? knew_row : vnew_row);
        uint4* dst = reinterpret_cast<uint4*>(lane < R4 ? kdst : vdst);
        dst[lane % R4] = src[lane % R4];
      }
      if (p.meta_pool != nullptr) {
        uint16_t* mn = p.meta_pool + (size_t)ph * 2 * D;
        uint16_t* mx = mn + D;
        for (int c = lane; c < D; c += kWave) {
          const uint16_t kb = knew_row[c];
          if (rn == 0) {
            mn[c] = kb;
            mx[c] = kb;
          } else {
            const float kf = bf16f(kb);
            if (kf < bf16f(mn[c])) mn[c] = kb;
            if (kf > bf16f(mx[c])) mx[c] = kb;
          }
        }
      }
      if (lane == 0) {
        p.pos_pool[(size_t)ph * kPage + rn] = p.new_pos[req];
        if (p.score_pool != nullptr) p.score_pool[(size_t)ph * kPage + rn] = 0.f;
      }
      __builtin_amdgcn_s_waitcnt(0);  // the stores are done before this wavefront reads the page
      // and no load of the page may be scheduled above them: the stream reads the
      // pool through other pointer types than the append writes it
      asm volatile("" ::: "memory");
    }
  }

  auto page_ref = [&](int i) -> PageRef {
    PageRef pr;
    const int gi = rbeg + wr + 4 * i;
    // wave-uniform by construction: keep them in scalar registers
    pr.vp = __builtin_amdgcn_readfirstlane(lds_vp[gi]);
    pr.lp = __builtin_amdgcn_readfirstlane(lds_lp[gi]);
    pr.phys = __builtin_amdgcn_readfirstlane(lds_phys[gi]);
    pr.nrows = __builtin_amdgcn_readfirstlane(min(kPage, Lp - pr.lp * kPage));
    pr.rn = -1;
    pr.tail = false;
    return pr;
  };

  // ---- the page stream.  K is prefetched two pages ahead (two register
  // buffers, pages alternate between them) and V one page ahead (one buffer):
  // page i+2's K loads are issued once page i's logits are formed, page i+1's
  // V loads once page i's PV is done.  The loads are unconditional (a
  // conditional load would make the compiler drain every load at the join);
  // past the last page they re-read one row of the last page.
  uint4 kbA[2 * K4], kbB[2 * K4];
  uint32_t vb[RPL];
  if (n_my > 0) {
    auto ref_or_tail = [&](int i) -> PageRef {
      PageRef r = page_ref(i < n_my ? i : n_my - 1);
      r.tail = i >= n_my;
      return r;
    };
    PageRef cur = ref_or_tail(0);
    PageRef nx1 = ref_or_tail(1);
    load_k<D>(p, ln, cur, kbA);
    __builtin_amdgcn_sched_barrier(0);
    load_k<D>(p, ln, nx1, kbB);
    __builtin_amdgcn_sched_barrier(0);
    load_v<D>(p, ln, cur, vb);
    for (int i = 0; i < n_my; i += 2) {
      {
        const PageRef nx2 = ref_or_tail(i + 2);
        float z[NP];
        qk_page<D, G>(ln, kbA, lds_q, z);
        load_k<D>(p, ln, nx2, kbA);
        softmax_page<D, G, W>(p, ln, cur, z, ws, lds_p[wave], lane, unit, ubase_p, lds_wh, lds_mr, wcap);
        pv_page<D, G>(ln, vb, cur.nrows, ws, lds_p[wave]);
        load_v<D>(p, ln, nx1, vb);
        cur = nx1;
        nx1 = nx2;
      }
      if (i + 1 >= n_my) break;
      {
        const PageRef nx2 = ref_or_tail(i + 3);
        float z[NP];
        qk_page<D, G>(ln, kbB, lds_q, z);
        load_k<D>(p, ln, nx2, kbB);
        softmax_page<D, G, W>(p, ln, cur, z, ws, lds_p[wave], lane, unit, ubase_p, lds_wh, lds_mr, wcap);
        pv_page<D, G>(ln, vb, cur.nrows, ws, lds_p[wave]);
        load_v<D>(p, ln, nx1, vb);
        cur = nx1;
        nx1 = nx2;
      }
    }
  }

  // ---- the fused steady eviction: this wavefront's slots' positions and old
  // scores are fetched now (every load in flight together; rows past the end
  // re-read a valid slot), while other wavefronts may still be streaming
  const bool steady_any = p.evict && p.accumulate && !quest && !bad && p.n_split == 1 && Lp == p.budget + 1 &&
                          Lp <= kMaxBudget && n_grp == g.n_visit;
  const bool steady = kWaveRows && steady_any && (max_rcnt + 3) / 4 <= 4 * kSteadyRows &&
                      g.n_visit <= kWeightPages<G, W>;
  int32_t spos[kSteadyRows];
  float su[kSteadyRows];
  if (kWaveRows && steady && n_my > 0) {
#pragma unroll
    for (int j = 0; j < kSteadyRows; ++j) {
      const int i = min((lane >> 4) + 4 * j, n_my - 1);
      const size_t a = (size_t)lds_phys[rbeg + wr + 4 * i] * kPage + (lane & (kPage - 1));
      spos[j] = p.pos_pool[a];
      su[j] = p.score_pool[a];
    }
  }

  // ---- per-wavefront totals into LDS
  float lsum[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    lsum[k] = ws.l_own[k];  // lanes of one head differ in lane bits 2..5
    lsum[k] += shfl_xor_f(lsum[k], 4);
    lsum[k] += shfl_xor_f(lsum[k], 8);
    lsum[k] += shfl_xor_f(lsum[k], 16);
    lsum[k] += shfl_xor_f(lsum[k], 32);
  }
  if (RS == 2) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      ws.o_acc[h][0] += shfl_xor_f(ws.o_acc[h][0], 32);
      ws.o_acc[h][1] += shfl_xor_f(ws.o_acc[h][1], 32);
    }
  }
  if (lane < GH) {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      lds_m[wave][lane + 4 * k] = ws.m_own[k];
      lds_l[wave][lane + 4 * k] = lsum[k];
    }
  }

  // ---- work-group partial (fixed wavefront order), GO heads per round.  A
  // unit's output and lse are stored at the very end of the kernel: a barrier
  // waits for the work-group's outstanding stores, which under a full memory
  // system take tens of microseconds.
  const bool single = p.n_split == 1;
  float* part_u = p.part + (size_t)unit * p.n_split * G * (D + 2);
  constexpr int OPR = (GO * D + NT - 1) / NT;  // outputs per thread and round
  constexpr int OPT = NRND * OPR;
  float out_v[OPT], lse_v[OPT];
#pragma unroll
  for (int k = 0; k < OPT; ++k) out_v[k] = lse_v[k] = 0.f;
#pragma unroll
  for (int rnd = 0; rnd < NRND; ++rnd) {
    if (rnd > 0) __syncthreads();  // the previous round's reads of lds_o
    if (lane < HP) {
#pragma unroll
      for (int h = 0; h < GO; ++h) {
        lds_o[wave][h][col] = ws.o_acc[rnd * GO + h][0];
        lds_o[wave][h][col + 1] = ws.o_acc[rnd * GO + h][1];
      }
    }
    __syncthreads();
    for (int idx = tid; idx < GO * D; idx += NT) {
      const int ho = idx / D;
      const int h = rnd * GO + ho;
      const int c = idx - ho * D;
      float ms = lds_m[0][h];
#pragma unroll
      for (int w = 1; w < NW; ++w) ms = fmaxf(ms, lds_m[w][h]);
      float o = 0.f, l = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float f = lds_m[w][h] == -INFINITY ? 0.f : fast_exp2(lds_m[w][h] - ms);
        o += lds_o[w][ho][c] * f;
        l += lds_l[w][h] * f;
      }
      if (single) {
        if (!bad) {
          out_v[rnd * OPR + (idx - tid) / NT] = o / l;
          if (c == 0) {
            lse_v[rnd * OPR + (idx - tid) / NT] = (ms + __log2f(l)) * kLn2;
            fin_m[h] = ms;
            fin_il[h] = 1.f / l;
          }
        }
      } else {
        float* rec = part_u + ((size_t)split * G + h) * (D + 2);
        if (c == 0) {
          rec[0] = ms;
          rec[1] = l;
        }
        rec[2 + c] = o;
      }
    }
  }

  if (!single) return;  // the combine kernel finishes the unit
  __syncthreads();
  if (bad) {
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    store_sel();
    return;
  }
  if (wcap > 0) {
    // each LDS page's reference maximum becomes the factor its weights take in
    // the score update, exp2(m_ref - m) / l per head: one exp2 per page and head
    // instead of per slot and head
    const int nl = min(g.n_visit, wcap) * G;
    for (int i = tid; i < nl; i += NT) {
      const int h = i % G;
      lds_mr[i] = fast_exp2(lds_mr[i] - fin_m[h]) * fin_il[h];
    }
    __syncthreads();
  }
  bool general;
  if (kWaveRows && steady) {
    const WeightSrc<W> wsrc{lds_wh, lds_mr, p.pbuf + ubase_p * kPage * G, p.mref + ubase_p * G, wcap};
    general = finish_steady<NT, G, D, W>(p, g, fin_m, fin_il, lds_phys, lds_vp, wsrc, spos, su, rbeg, wr, n_my,
                                         esc);
  } else if (!kWaveRows && steady_any) {
    const WeightSrc<W> wsrc{lds_wh, lds_mr, p.pbuf + ubase_p * kPage * G, p.mref + ubase_p * G, wcap};
    general = finish_steady_strided<NT, G, D, W>(p, g, fin_m, fin_il, lds_phys, wsrc, esc);
  } else {
    general = finish_unit<NT, G, !kQuest, W>(p, g, fin_m, fin_il, lds_wh, lds_mr, wcap);
  }
  if constexpr (!kQuest) {
    if (__builtin_expect(general, false)) evict_in_epilogue<NT, D>(p, g, esc);
  }
#pragma unroll
  for (int rnd = 0; rnd < NRND; ++rnd) {
#pragma unroll
    for (int k = 0; k < OPR; ++k) {
      const int idx = tid + k * NT;
      if (idx < GO * D) {
        const int ho = idx / D, c = idx - ho * D;
        const int h = rnd * GO + ho;
        p.out[((size_t)req * Hq + kvh * G + h) * D + c] = out_v[rnd * OPR + k];
        if (c == 0 && p.lse != nullptr) p.lse[(size_t)req * Hq + kvh * G + h] = lse_v[rnd * OPR + k];
      }
    }
  }
  store_sel();
}

// Launch order of the units when they take more than one round of work-groups:
// longest first (a counting sort on the page count), so that the last
// work-groups to start are the short ones and the chip drains evenly.  Units
// with equal page counts come in any order; the results do not depend on it.
constexpr int kOrderThreads = 1024;
constexpr int kOrderMaxBins = 16384;

__global__ __launch_bounds__(kOrderThreads) void unit_order_kernel(const int32_t* lengths, int num_units,
                                                                   int append, int max_pages, int32_t* order) {
  __shared__ int cnt[kOrderMaxBins];
  __shared__ int scan[kOrderThreads / kWave + 1];
  const int tid = threadIdx.x;
  const int nb = max_pages + 1;  // bin max_pages - pages: page counts 0..max_pages, descending
  auto bin_of = [&](int u) {
    const int L = lengths[u] + append;
    const int pages = L <= 0 ? 0 : min((L + kPage - 1) / kPage, max_pages);
    return max_pages - pages;
  };
  for (int i = tid; i < nb; i += kOrderThreads) cnt[i] = 0;
  __syncthreads();
  for (int u = tid; u < num_units; u += kOrderThreads) atomicAdd(&cnt[bin_of(u)], 1);
  __syncthreads();
  // exclusive scan over the bins: each thread sums a contiguous chunk
  const int chunk = (nb + kOrderThreads - 1) / kOrderThreads;
  const int c0 = min(nb, tid * chunk), c1 = min(nb, c0 + chunk);
  int local = 0;
  for (int i = c0; i < c1; ++i) local += cnt[i];
  int total;
  int run = block_exclusive_scan<kOrderThreads>(local, scan, &total);
  for (int i = c0; i < c1; ++i) {
    const int c = cnt[i];
    cnt[i] = run;
    run += c;
  }
  __syncthreads();
  for (int u = tid; u < num_units; u += kOrderThreads) order[atomicAdd(&cnt[bin_of(u)], 1)] = u;
}

// Second pass when a unit is split over several work-groups: combines the
// partials (m, l, o) in split order, writes out and lse, then finishes the unit.
constexpr int kCombineThreads = 512;

template <int D, int G>
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(const AttendParams p) {
  __shared__ float fin_m[G];
  __shared__ float fin_il[G];
  const UnitGeom g = unit_geom(p, blockIdx.x);
  if (g.bad) {
    if (threadIdx.x == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return;
  }
  const int Hq = p.hkv * G;
  const int n_act = min(p.n_split, ceil_div_dev(g.n_visit, p.pps));
  const float* part_u = p.part + (size_t)g.unit * p.n_split * G * (D + 2);
  for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
    const int h = idx / D;
    const int c = idx - h * D;
    float m = -INFINITY;
    for (int s = 0; s < n_act; ++s) m = fmaxf(m, part_u[((size_t)s * G + h) * (D + 2)]);
    float o = 0.f, l = 0.f;
    for (int s = 0; s < n_act; ++s) {
      const float* rec = part_u + ((size_t)s * G + h) * (D + 2);
      const float f = rec[0] == -INFINITY ? 0.f : fast_exp2(rec[0] - m);
      o += rec[2 + c] * f;
      l += rec[1] * f;
    }
    p.out[((size_t)g.req * Hq + g.kvh * G + h) * D + c] = o / l;
    if (c == 0) {
      if (p.lse != nullptr) p.lse[(size_t)g.req * Hq + g.kvh * G + h] = (m + __log2f(l)) * kLn2;
      fin_m[h] = m;
      fin_il[h] = 1.f / l;
    }
  }
  __syncthreads();
  finish_unit<kCombineThreads, G, false, float>(p, g, fin_m, fin_il, nullptr, nullptr, 0);
}

// With a split, the combine pass updates the scores and publishes the appended
// length; the eviction (if asked for) then runs as its own kernel, whose
// 1024-thread work-groups hold a whole long unit in registers.
// Units of at most this many pages take the per-wavefront steady eviction: the
// largest slot rank's share of them, over four wavefronts, fits kSteadyRows
// rows of four pages, and (finish_steady reads every page's weights from LDS)
// every page's weights fit the LDS buffer.
template <int NT, int G>
constexpr int wave_rows_pages() {
  constexpr int rows = (4 * 4 * kSteadyRows * 100 - 50) / RankWeights<NT / kWave / 4>::w[0];
  constexpr int lds = kWeightPages<G, WeightT<NT, true, G>>;
  return rows < lds ? rows : lds;
}
// groups of up to 4 are limited by the registers alone
static_assert(wave_rows_pages<kAttendThreads, 4>() == (4 * 4 * kSteadyRows * 100 - 50) / RankWeights<2>::w[0] &&
                  wave_rows_pages<kAttendThreadsWide, 4>() == (4 * 4 * kSteadyRows * 100 - 50) / RankWeights<4>::w[0],
              "per-wavefront steady eviction bounds");

// Launches with at most one work-group per compute unit take 1024 threads.
inline bool attend_wide(int num_units, int n_visit) {
  return (int64_t)num_units * ceil_div(n_visit, kMaxGroupPages) <= 256;
}

template <int D, int G, int NT>
static void launch_attend_nt(const AttendParams& prm, int grid, hipStream_t stream) {
  if (prm.sel != nullptr)  // Quest: no eviction code, per-wavefront rows are not used
    hipLaunchKernelGGL((decode_attend_kernel<D, G, NT, false, true>), dim3(grid), dim3(NT), 0, stream, prm);
  else if (prm.n_visit_max <= wave_rows_pages<NT, G>())
    hipLaunchKernelGGL((decode_attend_kernel<D, G, NT, true, false>), dim3(grid), dim3(NT), 0, stream, prm);
  else
    hipLaunchKernelGGL((decode_attend_kernel<D, G, NT, false, false>), dim3(grid), dim3(NT), 0, stream, prm);
}

template <int D, int G>
static void launch_attend(const AttendParams& prm, int grid, bool wide, hipStream_t stream) {
  if (wide)
    launch_attend_nt<D, G, kAttendThreadsWide>(prm, grid, stream);
  else
    launch_attend_nt<D, G, kAttendThreads>(prm, grid, stream);
  if (prm.n_split > 1) {
    AttendParams cp = prm;
    cp.evict = 0;
    const int units = grid / prm.n_split;
    hipLaunchKernelGGL((decode_combine_kernel<D, G>), dim3(units), dim3(kCombineThreads), 0, stream, cp);
    if (prm.evict) {
      EvictParams ep;
      ep.kv = const_cast<uint16_t*>(prm.kv);
      ep.pos_pool = prm.pos_pool;
      ep.score_pool = prm.score_pool;
      ep.block_table = prm.block_table;
      ep.lengths = prm.lengths;
      ep.num_pages = prm.num_pages;
      ep.max_pages = prm.max_pages;
      ep.budget = prm.budget;
      ep.recent = prm.recent;
      ep.max_len = prm.max_len;
      ep.freed_pages = prm.freed_pages;
      ep.freed_stride = prm.freed_stride;
      ep.freed_count = prm.freed_count;
      ep.dev_err = prm.dev_err;
      launch_evict(ep, units, D, stream);
    }
  }
}

}  // namespace se

using namespace se;

static int attend_n_visit(int32_t max_len, int32_t max_pages, int32_t top_k) {
  if (top_k > 0) return top_k + 1;
  int64_t ml = max_len;
  if (ml > (int64_t)max_pages * kPage) ml = (int64_t)max_pages * kPage;
  return (int)ceil_div(ml, kPage);
}

size_t se_attend_workspace_bytes(int32_t num_units, int32_t max_len, int32_t max_pages,
                                 int32_t q_per_kv, int32_t head_dim, int32_t top_k) {
  if (num_units <= 0 || max_len <= 0 || max_pages <= 0 || q_per_kv <= 0 || head_dim <= 0)
    return 0;
  const SplitShape s = split_shape(num_units, attend_n_visit(max_len, max_pages, top_k));
  return attend_ws_layout(num_units, s, q_per_kv, head_dim).total;
}

static se_status attend_launch(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                               const void* k_new, const void* v_new, const int32_t* new_pos,
                               const int32_t* sel_pages, int32_t top_k, float scale, int32_t max_len,
                               uint32_t flags, float* out, float* lse, float* logits,
                               int32_t logits_stride, void* ws, size_t ws_bytes, int32_t* dev_err,
                               hipStream_t stream, const AttendParams* fused_evict) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (q_per_kv != 1 && q_per_kv != 2 && q_per_kv != 4 && q_per_kv != 8) return SE_ERR_UNSUPPORTED;
  if (q == nullptr || out == nullptr || dev_err == nullptr || kv->kv_pool == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if ((k_new == nullptr) != (v_new == nullptr)) return SE_ERR_INVALID_ARGUMENT;
  if (k_new != nullptr && (new_pos == nullptr || kv->pos_pool == nullptr))
    return SE_ERR_INVALID_ARGUMENT;
  if (max_len <= 0) return SE_ERR_INVALID_ARGUMENT;
  if (sel_pages != nullptr) {
    if (top_k < 1 || top_k > 4096) return SE_ERR_INVALID_ARGUMENT;
    if (logits != nullptr) return SE_ERR_INVALID_ARGUMENT;
  } else {
    top_k = 0;
  }
  if ((flags & ~SE_ATTEND_ACCUMULATE) != 0) return SE_ERR_INVALID_ARGUMENT;
  const bool accumulate = (flags & SE_ATTEND_ACCUMULATE) != 0;
  if (accumulate && kv->score_pool == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (logits != nullptr && logits_stride < max_len) return SE_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f)) return SE_ERR_INVALID_ARGUMENT;

  const int D = kv->head_dim;
  const int n_visit = attend_n_visit(max_len, kv->max_pages, top_k);
  const bool wide = attend_wide(kv->num_units, n_visit);
  const SplitShape s = split_shape(kv->num_units, n_visit, wide ? 256 : 512);
  const AttendWs lay = attend_ws_layout(kv->num_units, s, q_per_kv, D);
  if (ws == nullptr || ws_bytes < lay.total) return SE_ERR_WORKSPACE;

  AttendParams prm = {};
  if (fused_evict != nullptr) prm = *fused_evict;
  prm.kv = static_cast<const uint16_t*>(kv->kv_pool);
  prm.pos_pool = kv->pos_pool;
  prm.score_pool = kv->score_pool;
  prm.meta_pool = static_cast<uint16_t*>(kv->meta_pool);
  prm.block_table = kv->block_table;
  prm.lengths = kv->lengths;
  prm.num_pages = kv->num_pages;
  prm.hkv = kv->num_kv_heads;
  prm.max_pages = kv->max_pages;
  prm.q = static_cast<const uint16_t*>(q);
  prm.k_new = static_cast<const uint16_t*>(k_new);
  prm.v_new = static_cast<const uint16_t*>(v_new);
  prm.new_pos = new_pos;
  prm.sel = sel_pages;
  prm.top_k = top_k;
  prm.scale = scale;
  prm.scale_log2 = scale * kLog2e;
  prm.max_len = max_len;
  prm.n_visit_max = s.n_visit;
  prm.pps = s.pps;
  prm.n_split = s.n_split;
  prm.accumulate = accumulate ? 1 : 0;
  prm.out = out;
  prm.lse = lse;
  prm.logits = logits;
  prm.logits_stride = logits_stride;
  char* base = static_cast<char*>(ws);
  prm.part = reinterpret_cast<float*>(base + lay.part);
  prm.pbuf = reinterpret_cast<float*>(base + lay.pbuf);
  prm.mref = reinterpret_cast<float*>(base + lay.mref);
  // more than one round of work-groups over ragged units: longest first
  prm.order = nullptr;
  if (sel_pages == nullptr && (int64_t)kv->num_units * s.n_split > (wide ? 256 : 512) &&
      kv->max_pages + 1 <= kOrderMaxBins) {
    int32_t* order = reinterpret_cast<int32_t*>(base + lay.order);
    hipLaunchKernelGGL(unit_order_kernel, dim3(1), dim3(kOrderThreads), 0, stream, kv->lengths, kv->num_units,
                       k_new != nullptr ? 1 : 0, kv->max_pages, order);
    prm.order = order;
  }
  prm.dev_err = dev_err;

  const int64_t grid = (int64_t)kv->num_units * s.n_split;
  if (grid > INT32_MAX) return SE_ERR_UNSUPPORTED;
  if (D == 128) {
    if (q_per_kv == 8) launch_attend<128, 8>(prm, (int)grid, wide, stream);
    else if (q_per_kv == 4) launch_attend<128, 4>(prm, (int)grid, wide, stream);
    else if (q_per_kv == 2) launch_attend<128, 2>(prm, (int)grid, wide, stream);
    else launch_attend<128, 1>(prm, (int)grid, wide, stream);
  } else {
    if (q_per_kv == 8) launch_attend<64, 8>(prm, (int)grid, wide, stream);
    else if (q_per_kv == 4) launch_attend<64, 4>(prm, (int)grid, wide, stream);
    else if (q_per_kv == 2) launch_attend<64, 2>(prm, (int)grid, wide, stream);
    else launch_attend<64, 1>(prm, (int)grid, wide, stream);
  }
  return launch_status();
}

extern "C" se_status se_decode_attend(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                                      const void* k_new, const void* v_new,
                                      const int32_t* new_pos, const int32_t* sel_pages,
                                      int32_t top_k, float scale, int32_t max_len,
                                      uint32_t flags, float* out, float* lse, float* logits,
                                      int32_t logits_stride, void* ws, size_t ws_bytes,
                                      int32_t* dev_err, hipStream_t stream) {
  return attend_launch(kv, q_per_kv, q, k_new, v_new, new_pos, sel_pages, top_k, scale, max_len,
                       flags, out, lse, logits, logits_stride, ws, ws_bytes, dev_err, stream,
                       nullptr);
}

extern "C" se_status se_decode_step_h2o(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                                        const void* k_new, const void* v_new,
                                        const int32_t* new_pos, float scale, int32_t budget,
                                        int32_t recent, int32_t max_len, float* out, float* lse,
                                        int32_t* freed_pages, int32_t freed_stride,
                                        int32_t* freed_count, void* ws, size_t ws_bytes,
                                        int32_t* dev_err, hipStream_t stream) {
  if (kv == nullptr || kv->score_pool == nullptr || kv->pos_pool == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if (budget < 1 || recent < 0) return SE_ERR_INVALID_ARGUMENT;
  if (budget > 8192) return SE_ERR_UNSUPPORTED;
  if (freed_pages != nullptr && freed_stride < kv->max_pages) return SE_ERR_INVALID_ARGUMENT;
  AttendParams ev = {};
  ev.evict = 1;
  ev.budget = budget;
  ev.recent = recent;
  ev.freed_pages = freed_pages;
  ev.freed_stride = freed_stride;
  ev.freed_count = freed_count;
  se_status st = attend_launch(kv, q_per_kv, q, k_new, v_new, new_pos, nullptr, 0, scale, max_len,
                               SE_ATTEND_ACCUMULATE, out, lse, nullptr, 0, ws, ws_bytes, dev_err,
                               stream, &ev);
  return st;
}

// ---- se_decode_step_h2o_noalloc: the same step with the workspace in a
// file-scope device array instead of a caller's buffer.  In host code the
// array's name is only a stand-in for the symbol: its device address (one per
// GPU, since every device loads its own copy of the code object) is looked up
// once per device with hipGetSymbolAddress and kept here.
constexpr size_t kStaticScratchBytes = size_t(256) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxScratchDevices] = {};

se_status static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SE_ERR_HIP;
  if (dev < 0 || dev >= kMaxScratchDevices) return SE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return SE_ERR_HIP;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return SE_OK;
}
}  // namespace

extern "C" size_t se_static_scratch_bytes(void) { return kStaticScratchBytes; }

extern "C" se_status se_decode_step_h2o_noalloc(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                                                const void* k_new, const void* v_new, const int32_t* new_pos,
                                                float scale, int32_t budget, int32_t recent, int32_t max_len,
                                                float* out, float* lse, int32_t* freed_pages, int32_t freed_stride,
                                                int32_t* freed_count, int32_t* dev_err, hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (max_len <= 0) return SE_ERR_INVALID_ARGUMENT;
  const size_t need = se_attend_workspace_bytes(kv->num_units, max_len, kv->max_pages, q_per_kv, kv->head_dim, 0);
  if (need > kStaticScratchBytes) return SE_ERR_WORKSPACE;
  void* ws = nullptr;
  st = static_scratch(&ws);
  if (st != SE_OK) return st;
  return se_decode_step_h2o(kv, q_per_kv, q, k_new, v_new, new_pos, scale, budget, recent, max_len, out, lse,
                            freed_pages, freed_stride, freed_count, ws, kStaticScratchBytes, dev_err, stream);
}

size_t se_quest_step_workspace_bytes(int32_t num_units, int32_t max_len, int32_t max_pages, int32_t q_per_kv,
                                     int32_t head_dim, int32_t top_k) {
  const size_t a = se_attend_workspace_bytes(num_units, max_len, max_pages, q_per_kv, head_dim, top_k);
  if (a == 0) return 0;
  return a + se_quest_workspace_bytes(num_units, max_pages);
}

extern "C" se_status se_decode_step_quest(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                                          const void* k_new, const void* v_new, const int32_t* new_pos,
                                          float scale, int32_t top_k, int32_t max_len, int32_t* sel_pages,
                                          float* out, float* lse, void* ws, size_t ws_bytes, int32_t* dev_err,
                                          hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->meta_pool == nullptr || sel_pages == nullptr || q == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (top_k < 1 || top_k > 4096 || max_len < 1) return SE_ERR_INVALID_ARGUMENT;
  const size_t a_bytes =
      se_attend_workspace_bytes(kv->num_units, max_len, kv->max_pages, q_per_kv, kv->head_dim, top_k);
  if (ws == nullptr || ws_bytes < a_bytes) return SE_ERR_WORKSPACE;
  // one launch when one work-group holds each unit and the candidates fit LDS
  const int n_visit = top_k + 1;
  const bool wide = attend_wide(kv->num_units, n_visit);
  const SplitShape s = split_shape(kv->num_units, n_visit, wide ? 256 : 512);
  int64_t ml = max_len;
  if (ml > (int64_t)kv->max_pages * kPage) ml = (int64_t)kv->max_pages * kPage;
  if (s.n_split == 1 && ml / kPage + top_k <= kSelectMaxPages) {
    AttendParams ex = {};
    ex.select = 1;
    ex.meta = static_cast<const uint16_t*>(kv->meta_pool);
    return attend_launch(kv, q_per_kv, q, k_new, v_new, new_pos, sel_pages, top_k, scale, max_len, 0, out, lse,
                         nullptr, 0, ws, ws_bytes, dev_err, stream, &ex);
  }
  // otherwise the two calls; the selection's workspace follows the attention's
  char* base = static_cast<char*>(ws);
  st = se_quest_select(kv, q_per_kv, q, scale, top_k, max_len, 0, sel_pages, nullptr, 0, base + a_bytes,
                       ws_bytes - a_bytes, dev_err, stream);
  if (st != SE_OK) return st;
  return attend_launch(kv, q_per_kv, q, k_new, v_new, new_pos, sel_pages, top_k, scale, max_len, 0, out, lse,
                       nullptr, 0, ws, ws_bytes, dev_err, stream, nullptr);
}
