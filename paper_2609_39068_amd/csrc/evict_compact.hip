// se_evict_compact: H2O retention (Appendix A.3, eq. background-h2o-retention) and
// in-place compaction of the retained slots (Section 3.1), one 1024-thread
// work-group per unit running evict_unit_wide (evict_core.h, which describes the
// selection and the compaction).  se_decode_step_h2o launches the same kernel
// after its combine pass when a unit's attention was split.
#include "evict_core.h"

namespace se {

constexpr int kEvictThreads = 1024;
constexpr int kEvictSlotsPerThread = 34;  // register-resident up to 40960 slots per unit

template <int D>
__global__ __launch_bounds__(kEvictThreads) void evict_compact_kernel(const EvictParams p) {
  SE_WIDE_SCRATCH(kEvictThreads, kEvictSlotsPerThread, sc);
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
  evict_unit_wide<kEvictThreads, D, kEvictSlotsPerThread>(job, sc);
}

void launch_evict(const EvictParams& p, int num_units, int head_dim, hipStream_t stream) {
  if (head_dim == 128)
    hipLaunchKernelGGL((evict_compact_kernel<128>), dim3(num_units), dim3(kEvictThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((evict_compact_kernel<64>), dim3(num_units), dim3(kEvictThreads), 0, stream, p);
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

