// se_evict_compact: H2O retention (Appendix A.3, eq. background-h2o-retention) and
// in-place compaction of the retained slots (Section 3.1), one 1024-thread
// work-group per unit running evict_unit_wide (evict_core.h, which describes the
// selection and the compaction).  se_decode_step_h2o launches the same kernel
// after its combine pass when a unit's attention was split.
#include <algorithm>

#include "evict_core.h"

namespace se {

constexpr int kEvictThreads = 1024;
constexpr int kEvictSlotsPerThread = 34;  // register-resident up to 40960 slots per unit

template <int D>
__global__ __launch_bounds__(kEvictThreads) void evict_compact_kernel(const EvictParams p) {
  SE_WIDE_SCRATCH(kEvictThreads, kEvictSlotsPerThread, sc);
  int32_t* const moves = p.moves != nullptr ? p.moves + (size_t)blockIdx.x * kMoveListInts : nullptr;
  if (moves != nullptr && threadIdx.x == 0) moves[0] = 0;  // every path that moves nothing leaves 0
  EvictJob job;
  job.kv = p.kv;
  job.pos_pool = p.pos_pool;
  job.score_pool = p.score_pool;
  job.bt = p.block_table + (size_t)blockIdx.x * p.max_pages;
  job.lengths = p.lengths;
  job.num_pages = p.num_pages;
  job.unit = blockIdx.x;
  job.L = p.lengths[blockIdx.x];
  job.budget = p.budget;
  job.recent = p.recent;
  job.max_len = p.max_len;
  job.max_pages = p.max_pages;
  job.freed_pages = p.freed_pages;
  job.freed_stride = p.freed_stride;
  job.freed_count = p.freed_count;
  job.dev_err = p.dev_err;
  job.moves = moves;
  evict_unit_wide<kEvictThreads, D, kEvictSlotsPerThread>(job, sc);
}

constexpr int kMoveThreads = 256;
constexpr int kMoveGroups = 2048;  // work-groups the moves of a launch are spread over

// The deferred moves of evict_compact_kernel: work-group (unit, split) moves
// the unit's movers r = split * MPP + m + k * splits * MPP into their holes with
// key row, value row, position and score, one 16-byte chunk per thread, four
// movers in flight.  Holes and movers are disjoint, so the moves are
// independent; the kernel boundary orders them after every unit's selection.
template <int D>
__global__ __launch_bounds__(kMoveThreads) void evict_move_kernel(const EvictParams p, int splits) {
  constexpr int C = D / 8;        // chunks per row
  constexpr int TPM = 2 * C;      // threads per mover (key row, then value row)
  constexpr int MPP = kMoveThreads / TPM;
  const int unit = blockIdx.x;
  const int32_t* ml = p.moves + (size_t)unit * kMoveListInts;
  const int n = ml[0];
  if (n <= 0) return;
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int c = threadIdx.x % TPM;
  const int off = (c < C ? 0 : kPage * D) + (c % C) * 8;  // in bf16 elements
  int32_t* const side = c == 0 ? p.pos_pool : reinterpret_cast<int32_t*>(p.score_pool);
  auto row = [&](int s) -> uint4* {
    return reinterpret_cast<uint4*>(p.kv + (size_t)bt[s >> 4] * 2 * kPage * D + (s & (kPage - 1)) * D + off);
  };
  auto addr = [&](int s) -> size_t { return (size_t)bt[s >> 4] * kPage + (s & (kPage - 1)); };
  const int step = splits * MPP;
  int r = blockIdx.y * MPP + (int)threadIdx.x / TPM;
  for (; r + 3 * step < n; r += 4 * step) {
    const int s0 = ml[kMoveMovers + r], s1 = ml[kMoveMovers + r + step], s2 = ml[kMoveMovers + r + 2 * step],
              s3 = ml[kMoveMovers + r + 3 * step];
    const int d0 = ml[kMoveHoles + r], d1 = ml[kMoveHoles + r + step], d2 = ml[kMoveHoles + r + 2 * step],
              d3 = ml[kMoveHoles + r + 3 * step];
    const uint4 v0 = *row(s0), v1 = *row(s1), v2 = *row(s2), v3 = *row(s3);
    int32_t x0 = 0, x1 = 0, x2 = 0, x3 = 0;
    if (c < 2) {
      x0 = side[addr(s0)];
      x1 = side[addr(s1)];
      x2 = side[addr(s2)];
      x3 = side[addr(s3)];
    }
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
  for (; r < n; r += step) {
    const int s0 = ml[kMoveMovers + r], d0 = ml[kMoveHoles + r];
    const uint4 v0 = *row(s0);
    int32_t x0 = 0;
    if (c < 2) x0 = side[addr(s0)];
    *row(d0) = v0;
    if (c < 2) side[addr(d0)] = x0;
  }
}

// Below one unit per CU the selection kernel leaves most of the chip idle, and
// the moves, spread over many work-groups, go faster on their own; with more
// units, each work-group's moves overlap the other work-groups' selections
// (measured: 64 units of 10240 slots, 69 -> 59 us; 512 units of 32768 slots,
// 482 -> 539 us deferred).
constexpr int kDeferMovesBelowUnits = 256;

void launch_evict(const EvictParams& prm, int num_units, int head_dim, hipStream_t stream) {
  EvictParams p = prm;
  if (num_units >= kDeferMovesBelowUnits) p.moves = nullptr;
  if (head_dim == 128)
    hipLaunchKernelGGL((evict_compact_kernel<128>), dim3(num_units), dim3(kEvictThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((evict_compact_kernel<64>), dim3(num_units), dim3(kEvictThreads), 0, stream, p);
  if (p.moves == nullptr) return;
  const int splits = std::max(1, std::min(32, (int)ceil_div(kMoveGroups, num_units)));
  if (head_dim == 128)
    hipLaunchKernelGGL((evict_move_kernel<128>), dim3(num_units, splits), dim3(kMoveThreads), 0, stream, p, splits);
  else
    hipLaunchKernelGGL((evict_move_kernel<64>), dim3(num_units, splits), dim3(kMoveThreads), 0, stream, p, splits);
}

}  // namespace se

using namespace se;

extern "C" se_status se_evict_compact(const se_kv_view* kv, int32_t budget, int32_t recent,
                                      int32_t max_len, int32_t* freed_pages,
                                      int32_t freed_stride, int32_t* freed_count,
                                      int32_t* dev_err, hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->kv_pool == nullptr || kv->pos_pool == nullptr || kv->score_pool == nullptr ||
      dev_err == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if (budget < 1 || recent < 0 || max_len < 1) return SE_ERR_INVALID_ARGUMENT;
  if (budget > kMaxBudget) return SE_ERR_UNSUPPORTED;
  if (freed_pages != nullptr && freed_stride < kv->max_pages) return SE_ERR_INVALID_ARGUMENT;
  EvictParams prm;
  prm.kv = static_cast<uint16_t*>(kv->kv_pool);
  prm.pos_pool = kv->pos_pool;
  prm.score_pool = kv->score_pool;
  prm.block_table = kv->block_table;
  prm.lengths = kv->lengths;
  prm.num_pages = kv->num_pages;
  prm.max_pages = kv->max_pages;
  prm.budget = budget;
  prm.recent = recent;
  prm.max_len = max_len;
  prm.freed_pages = freed_pages;
  prm.freed_stride = freed_stride;
  prm.freed_count = freed_count;
  prm.dev_err = dev_err;
  launch_evict(prm, kv->num_units, kv->head_dim, stream);
  return launch_status();
}

