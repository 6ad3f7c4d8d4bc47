// se_prune_interval: sparsity-based prefix-cache pruning of a history interval
// (Section 3.2, "Sparsity-Based Prefix-Cache Pruning", eq. prefix-pruning;
// Appendix C.2, "Pruning Metadata and Cache Operations").  With T the logical
// positions [lo, hi) of a unit and I the positions of T a policy keeps, the
// unit's resident set becomes (R minus T) union I; positions are not renumbered.
//
// One 256-thread work-group per unit:
//   1. The unit's block-table row goes to LDS (entries checked); one pass over
//      the positions counts the interval's resident slots and finds the first
//      and last of them.
//   2. Budget mode: an 8-bit radix selection over 64-bit keys (order-preserving
//      score bits, then the inverted position bits, so equal scores keep the
//      lower position) of the interval's slots, within the slot range found in
//      step 1, gives the threshold of the budget largest.  Mask mode: a slot of
//      the interval stays iff its mask byte (at position - lo) is nonzero.
//   3. Order-keeping compaction from the interval's first slot on, 64 slots a
//      round: every wavefront evaluates the round's 64 keep flags (one slot per
//      lane) and ballots them, so each lane knows the rank of every slot of the
//      round without LDS.  The moving slots' rows are loaded as 16-byte pieces
//      (a slot's key and value rows are 4*D bytes), the work-group meets at a
//      barrier once every load of the round has returned -- a destination can
//      be a source of the same round -- and the pieces, positions and scores
//      are stored at their ranks.  A destination is never above its source and
//      later rounds read only slots above this round, so the next round's loads
//      never meet this round's stores.
//   4. The pages past the new length are reported, the length written, and the
//      Quest summaries (when the view has them) of the pages from the
//      interval's first slot on are rebuilt from the stored keys.
#include <climits>

#include "se_common.h"

namespace se {

constexpr int kPruneThreads = 256;
constexpr int kPruneMaxPages = 8192;   // 131072 slots per unit
constexpr int kPruneRound = kWave;     // slots per compaction round
constexpr int kPruneBatch = 8;         // positions in flight per thread in the scans

struct PruneParams {
  uint16_t* kv;
  int32_t* pos_pool;
  float* score_pool;
  uint16_t* meta_pool;
  const int32_t* block_table;
  int32_t* lengths;
  int64_t num_pages;
  int32_t max_pages;
  const int32_t* interval;   // [num_units][2]: lo, hi
  const uint8_t* keep_mask;  // [num_units][mask_stride] or NULL
  int32_t mask_stride;
  const int32_t* keep_budget;  // [num_units] or NULL
  int32_t max_len;
  int32_t* freed_pages;
  int32_t freed_stride;
  int32_t* freed_count;
  int32_t* dev_err;
};

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Selection key: larger keeps first; equal scores keep the lower position.
__device__ __forceinline__ uint64_t prune_key(float score, int32_t pos) {
  return ((uint64_t)float_key(score) << 32) | (uint64_t)(~((uint32_t)pos ^ 0x80000000u));
}

template <int D>
__global__ __launch_bounds__(kPruneThreads, 4) void prune_interval_kernel(const PruneParams p) {
  constexpr int NT = kPruneThreads;
  constexpr int PPS = 4 * D / 16;            // 16-byte pieces of a slot's key and value rows
  constexpr int KP = D / 8;                  // of them in the key row
  constexpr int SPK = NT / PPS;              // slots covered by one piece per thread
  constexpr int KPT = kPruneRound / SPK;     // pieces per thread per round
  static_assert(KPT * SPK == kPruneRound, "whole slots per round");
  __shared__ int s_bt[kPruneMaxPages];
  __shared__ unsigned s_hist[256];
  __shared__ int s_scan[NT / kWave + 1];
  __shared__ int s_bcast[4];
  __shared__ int s_red[NT / kWave];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int unit = blockIdx.x;
  const int L = p.lengths[unit];
  if (L < 0 || L > p.max_len || L > p.max_pages * kPage || L > kPruneMaxPages * kPage) {
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return;
  }
  const int lo = p.interval[2 * unit];
  const int hi = p.interval[2 * unit + 1];
  const bool by_mask = p.keep_mask != nullptr;
  const int budget = by_mask ? 0 : p.keep_budget[unit];
  if ((by_mask && (int64_t)hi - lo > (int64_t)p.mask_stride) || budget < 0) {
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_INTERVAL);
    return;
  }
  const int n_pages = ceil_div_dev(L, kPage);
  {
    int bad = 0;
    for (int i = tid; i < n_pages; i += NT) {
      const int ph = p.block_table[(size_t)unit * p.max_pages + i];
      bad |= (ph < 0 || (int64_t)ph >= p.num_pages);
      s_bt[i] = ph;
    }
    bad = block_reduce<NT>(bad, s_red, [](int a, int b) { return a | b; });
    if (bad) {
      if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
      return;
    }
  }
  auto slot_addr = [&](int s) { return (size_t)s_bt[s >> 4] * kPage + (s & (kPage - 1)); };
  auto in_t = [&](int32_t ps) { return ps >= lo && ps < hi; };
  auto no_change = [&]() {
    if (tid == 0 && p.freed_count != nullptr) p.freed_count[unit] = 0;
  };

  // ---- 1. the interval's resident slots: count, first and last slot
  int cnt = 0, first = INT_MAX, last = -1;
  for (int b = tid; b < L; b += NT * kPruneBatch) {
    int32_t ps[kPruneBatch];
#pragma unroll
    for (int k = 0; k < kPruneBatch; ++k) {
      const int s = b + k * NT;
      ps[k] = s < L ? p.pos_pool[slot_addr(s)] : INT_MIN;
    }
#pragma unroll
    for (int k = 0; k < kPruneBatch; ++k) {
      const int s = b + k * NT;
      if (s < L && in_t(ps[k])) {
        ++cnt;
        first = min(first, s);
        last = max(last, s);
      }
    }
  }
  cnt = block_reduce<NT>(cnt, s_red, [](int a, int b) { return a + b; });
  first = block_reduce<NT>(first, s_red, [](int a, int b) { return min(a, b); });
  last = block_reduce<NT>(last, s_red, [](int a, int b) { return max(a, b); });
  if (cnt == 0 || (!by_mask && budget >= cnt)) {  // nothing of the interval leaves
    no_change();
    return;
  }

  // ---- 2. budget mode: threshold of the budget largest keys among the interval's slots
  const bool keep_none = !by_mask && budget == 0;
  uint64_t kprefix = 0, kmask = 0;
  if (!by_mask && budget > 0) {
    uint64_t prefix = 0, mask = 0;
    int k = budget;
    for (int shift = 56; shift >= 0; shift -= 8) {
      s_hist[tid] = 0;  // NT == 256 bins
      __syncthreads();
      for (int b = first + tid; b <= last; b += NT * kPruneBatch) {
        int32_t ps[kPruneBatch];
        float sc[kPruneBatch];
#pragma unroll
        for (int j = 0; j < kPruneBatch; ++j) {
          const int s = b + j * NT;
          ps[j] = INT_MIN;
          sc[j] = 0.f;
          if (s <= last) {
            const size_t a = slot_addr(s);
            ps[j] = p.pos_pool[a];
            sc[j] = p.score_pool[a];
          }
        }
#pragma unroll
        for (int j = 0; j < kPruneBatch; ++j) {
          const int s = b + j * NT;
          if (s > last || !in_t(ps[j])) continue;
          const uint64_t key = prune_key(sc[j], ps[j]);
          if ((key & mask) == prefix) atomicAdd(&s_hist[(unsigned)(key >> shift) & 255u], 1u);
        }
      }
      __syncthreads();
      const int v = (int)s_hist[255 - tid];  // thread t counts digit 255 - t
      int total;
      const int excl = block_exclusive_scan<NT>(v, s_scan, &total);
      if (v > 0 && excl < k && excl + v >= k) {
        s_bcast[0] = 255 - tid;
        s_bcast[1] = excl;
        s_bcast[2] = v;
      }
      __syncthreads();
      const int d = s_bcast[0];
      k -= s_bcast[1];
      const int c = s_bcast[2];
      __syncthreads();
      prefix |= (uint64_t)d << shift;
      mask |= (uint64_t)0xFF << shift;
      if (c == k) break;  // every key with this prefix is kept
    }
    kprefix = prefix;
    kmask = mask;
  }

  // ---- 3. order-keeping compaction from the round holding the first interval slot
  const uint8_t* kmrow = by_mask ? p.keep_mask + (size_t)unit * p.mask_stride : nullptr;
  const int r0 = first & ~(kPruneRound - 1);
  int base = r0;  // slots kept below the round: every slot below `first` stays in place
  // A lane's keep flag needs its slot's position, then the mask byte at that
  // position (or the slot's score): both are fetched ahead -- the position two
  // rounds ahead, the second input one round ahead -- so that a round waits
  // only for its own rows.  Those slots are above every destination written
  // before their round, so the values read are the ones the round decides on.
  auto load_pos = [&](int s) -> int32_t { return s < L ? p.pos_pool[slot_addr(s)] : INT_MIN; };
  auto load_aux = [&](int s, int32_t ps) -> float {
    if (s >= L || !in_t(ps)) return 0.f;
    if (by_mask) return (float)kmrow[(int64_t)ps - lo];
    return keep_none ? 0.f : p.score_pool[slot_addr(s)];
  };
  auto keep_of = [&](int s, int32_t ps, float aux) -> bool {
    if (s >= L) return false;
    if (!in_t(ps)) return true;
    if (by_mask) return aux != 0.f;
    return !keep_none && (prune_key(aux, ps) & kmask) >= kprefix;
  };
  int32_t pos0 = load_pos(r0 + lane);
  float aux0 = load_aux(r0 + lane, pos0);
  int32_t pos1 = load_pos(r0 + kPruneRound + lane);
  for (int c0 = r0; c0 < L; c0 += kPruneRound) {
    const bool keep = keep_of(c0 + lane, pos0, aux0);
    const float aux1 = load_aux(c0 + kPruneRound + lane, pos1);
    const int32_t pos2 = load_pos(c0 + 2 * kPruneRound + lane);
    const uint64_t bits = __builtin_amdgcn_ballot_w64(keep);  // the same in every wavefront
    const int n_keep = __popcll(bits);
    pos0 = pos1;
    aux0 = aux1;
    pos1 = pos2;
    if (bits == (n_keep == 64 ? ~0ull : ((1ull << n_keep) - 1)) && base == c0) {
      base += n_keep;  // the round's kept slots are its first ones and already in place
      continue;
    }
    u32x4_t buf[KPT];
    int dst[KPT];
    int32_t mpos[KPT];
    float mscore[KPT];
    const int pc = tid % PPS;
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const int j = tid / PPS + SPK * k;
      const int s = c0 + j;
      const bool kept = (bits >> j) & 1ull;
      const int d = base + __popcll(bits & ((1ull << j) - 1ull));
      dst[k] = (kept && d != s) ? d : -1;
      buf[k] = u32x4_t{0u, 0u, 0u, 0u};
      mpos[k] = 0;
      mscore[k] = 0.f;
      if (dst[k] >= 0) {
        const uint16_t* pg = p.kv + (size_t)s_bt[s >> 4] * 2 * kPage * D;
        const int row = s & (kPage - 1);
        const uint16_t* src = pc < KP ? pg + row * D + pc * 8 : pg + kPage * D + row * D + (pc - KP) * 8;
        buf[k] = *reinterpret_cast<const u32x4_t*>(src);
        if (pc == 0) mpos[k] = p.pos_pool[slot_addr(s)];
        if (pc == 1 && p.score_pool != nullptr) mscore[k] = p.score_pool[slot_addr(s)];
      }
    }
    // every load of the round has returned before any store of it
#pragma unroll
    for (int k = 0; k < KPT; ++k)
      asm volatile("" ::"v"(buf[k].x), "v"(buf[k].y), "v"(buf[k].z), "v"(buf[k].w), "v"(mpos[k]), "v"(mscore[k]));
    __syncthreads();
#pragma unroll
    for (int k = 0; k < KPT; ++k) {
      const int d = dst[k];
      if (d < 0) continue;
      uint16_t* pg = p.kv + (size_t)s_bt[d >> 4] * 2 * kPage * D;
      const int row = d & (kPage - 1);
      uint16_t* out = pc < KP ? pg + row * D + pc * 8 : pg + kPage * D + row * D + (pc - KP) * 8;
      *reinterpret_cast<u32x4_t*>(out) = buf[k];
      if (pc == 0) p.pos_pool[slot_addr(d)] = mpos[k];
      if (pc == 1 && p.score_pool != nullptr) p.score_pool[slot_addr(d)] = mscore[k];
    }
    base += n_keep;
  }
  const int Lp = base;

  // ---- 4. released pages, the new length, Quest summaries of the changed pages
  const int f0 = ceil_div_dev(Lp, kPage);
  const int nf = n_pages - f0;
  if (p.freed_pages != nullptr)
    for (int i = tid; i < nf; i += NT) p.freed_pages[(size_t)unit * p.freed_stride + i] = s_bt[f0 + i];
  if (tid == 0) {
    if (p.freed_count != nullptr) p.freed_count[unit] = nf;
    p.lengths[unit] = Lp;
  }
  if (p.meta_pool != nullptr && first < Lp) {
    __syncthreads();  // the compaction's stores are visible to every wavefront
    const int wave = tid / kWave;
    for (int lp = first / kPage + wave; lp < f0; lp += NT / kWave) {
      if (lane >= D / 2) continue;
      const int nrows = min(kPage, Lp - lp * kPage);
      const uint16_t* kpage = p.kv + (size_t)s_bt[lp] * 2 * kPage * D;
      uint32_t w = *reinterpret_cast<const uint32_t*>(kpage + 2 * lane);
      uint32_t mn0 = w & 0xffffu, mx0 = mn0, mn1 = w >> 16, mx1 = mn1;
      for (int r = 1; r < nrows; ++r) {
        w = *reinterpret_cast<const uint32_t*>(kpage + r * D + 2 * lane);
        const uint32_t a = w & 0xffffu, b = w >> 16;
        if (bf16f((uint16_t)a) < bf16f((uint16_t)mn0)) mn0 = a;
        if (bf16f((uint16_t)a) > bf16f((uint16_t)mx0)) mx0 = a;
        if (bf16f((uint16_t)b) < bf16f((uint16_t)mn1)) mn1 = b;
        if (bf16f((uint16_t)b) > bf16f((uint16_t)mx1)) mx1 = b;
      }
      uint16_t* meta = p.meta_pool + (size_t)s_bt[lp] * 2 * D;
      *reinterpret_cast<uint32_t*>(meta + 2 * lane) = mn0 | (mn1 << 16);
      *reinterpret_cast<uint32_t*>(meta + D + 2 * lane) = mx0 | (mx1 << 16);
    }
  }
}

}  // namespace se

using namespace se;

extern "C" se_status se_prune_interval(const se_kv_view* kv, const int32_t* interval, const uint8_t* keep_mask,
                                       int32_t mask_stride, const int32_t* keep_budget, int32_t max_len,
                                       int32_t* freed_pages, int32_t freed_stride, int32_t* freed_count,
                                       int32_t* dev_err, hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->kv_pool == nullptr || kv->pos_pool == nullptr || interval == nullptr || dev_err == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if ((keep_mask == nullptr) == (keep_budget == nullptr)) return SE_ERR_INVALID_ARGUMENT;
  if (keep_mask != nullptr && mask_stride < 1) return SE_ERR_INVALID_ARGUMENT;
  if (keep_budget != nullptr && kv->score_pool == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (max_len < 1) return SE_ERR_INVALID_ARGUMENT;
  if (max_len > kPruneMaxPages * kPage) return SE_ERR_UNSUPPORTED;
  if (freed_pages != nullptr && freed_stride < kv->max_pages) return SE_ERR_INVALID_ARGUMENT;
  PruneParams prm;
  prm.kv = static_cast<uint16_t*>(kv->kv_pool);
  prm.pos_pool = kv->pos_pool;
  prm.score_pool = kv->score_pool;
  prm.meta_pool = static_cast<uint16_t*>(kv->meta_pool);
  prm.block_table = kv->block_table;
  prm.lengths = kv->lengths;
  prm.num_pages = kv->num_pages;
  prm.max_pages = kv->max_pages;
  prm.interval = interval;
  prm.keep_mask = keep_mask;
  prm.mask_stride = mask_stride;
  prm.keep_budget = keep_budget;
  prm.max_len = max_len;
  prm.freed_pages = freed_pages;
  prm.freed_stride = freed_stride;
  prm.freed_count = freed_count;
  prm.dev_err = dev_err;
  if (kv->head_dim == 128)
    hipLaunchKernelGGL((prune_interval_kernel<128>), dim3(kv->num_units), dim3(kPruneThreads), 0, stream, prm);
  else
    hipLaunchKernelGGL((prune_interval_kernel<64>), dim3(kv->num_units), dim3(kPruneThreads), 0, stream, prm);
  return launch_status();
}
