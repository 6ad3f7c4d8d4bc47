// Quest page summaries and query-dependent page selection (Appendix A.3,
// eqs. background-quest-summary and background-quest-score).
//
// se_quest_summarize: one wavefront per page, lane pairs of columns, running
// min/max over the page's resident rows (exact on bf16 values).
//
// se_quest_select, two kernels:
//   * bound: 8 lanes share one page (16 for groups of 8 at D = 128), each
//     owning D/8 (D/16) channels of the page's min and max rows (16-byte
//     loads).  max(q*m, q*M) = q+ * M + q- * m with q+ = max(q, 0) and
//     q- = min(q, 0) (one of the two products is an exact zero), so the bound
//     is two bf16 pair dot products per channel pair and needs no per-channel
//     branch.  A 3-step (4-step) lane reduction gives the page's bound per
//     query row; the page score is the maximum over the G rows.
//   * top-k: one work-group per unit, radix selection on order-preserving
//     integer keys of the scores; equal scores keep the lower page index; the
//     selected pages are written in ascending order by a block scan.
// With at least one unit per compute unit (and at most kFusedMaxPages
// candidates), one 1024-thread work-group per unit does both: the unit's
// block-table row and its page scores stay in LDS, the bounds stream at the
// compute unit's full rate, and the selection runs on the LDS scores (same
// arithmetic and the same selection as the two kernels).
#include <climits>

#include "quest_core.h"

namespace se {

struct QuestParams {
  const uint16_t* kv;
  uint16_t* meta_pool;
  const int32_t* block_table;
  const int32_t* lengths;
  int64_t num_pages;
  int32_t hkv;
  int32_t max_pages;
  int32_t max_len;
  const uint16_t* q;
  float scale;
  int32_t top_k;
  int32_t* sel;
  float* scores;
  int32_t scores_stride;
  int32_t blocks_per_unit;
  int32_t write_scores;  // fused kernel: also store the page scores
  int32_t* dev_err;
};

__device__ __forceinline__ bool unit_length_ok(const QuestParams& p, int L) {
  return L >= 0 && L <= p.max_len && L <= p.max_pages * kPage;
}

template <int D>
__global__ __launch_bounds__(256) void quest_summarize_kernel(const QuestParams p) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int unit = blockIdx.x / p.blocks_per_unit;
  const int lp = (blockIdx.x - unit * p.blocks_per_unit) * 4 + wave;
  const int L = p.lengths[unit];
  if (!unit_length_ok(p, L)) {
    if (threadIdx.x == 0 && blockIdx.x % p.blocks_per_unit == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return;
  }
  if (lp * kPage >= L) return;
  const int phys = p.block_table[(size_t)unit * p.max_pages + lp];
  if (phys < 0 || (int64_t)phys >= p.num_pages) {
    if (lane == 0) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
    return;
  }
  if (lane >= D / 2) return;
  const int nrows = min(kPage, L - lp * kPage);
  const uint16_t* kpage = p.kv + (size_t)phys * 2 * kPage * D;
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
  uint16_t* meta = p.meta_pool + (size_t)phys * 2 * D;
  *reinterpret_cast<uint32_t*>(meta + 2 * lane) = mn0 | (mn1 << 16);
  *reinterpret_cast<uint32_t*>(meta + D + 2 * lane) = mx0 | (mx1 << 16);
}

constexpr int kBoundPagesPerGroup = 256;

template <int D, int G>
__global__ __launch_bounds__(256) void quest_bound_kernel(const QuestParams p) {
  using BL = BoundLanes<D, G>;
  constexpr int CH = BL::CH, CW = BL::CW, C4 = BL::C4, LPP = BL::LPP;
  constexpr int PPI = 256 / LPP;  // pages per iteration of the work-group
  const int lane = threadIdx.x & 63;
  const int g = lane & (LPP - 1);
  const int unit = blockIdx.x / p.blocks_per_unit;
  const int chunk = blockIdx.x - unit * p.blocks_per_unit;
  const int req = unit / p.hkv;
  const int kvh = unit - req * p.hkv;
  const int L = p.lengths[unit];
  if (!unit_length_ok(p, L)) return;  // reported by the top-k kernel
  const int n_cand = L / kPage;
  const int b0 = chunk * kBoundPagesPerGroup;
  if (b0 >= n_cand) return;
  const int b1 = min(b0 + kBoundPagesPerGroup, n_cand);

  uint32_t qp[G][CW], qn[G][CW];
  bound_query<D, G>(p.q + ((size_t)req * p.hkv * G + (size_t)kvh * G) * D, g, qp, qn);

  for (int b = b0 + (int)threadIdx.x / LPP; b < b0 + kBoundPagesPerGroup; b += PPI) {
    const bool valid = b < b1;
    if (__ballot(valid) == 0) break;
    int phys = 0;
    if (valid) {
      phys = p.block_table[(size_t)unit * p.max_pages + b];
      if (phys < 0 || (int64_t)phys >= p.num_pages) {
        set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
        phys = -1;
      }
    }
    const bool load = valid && phys >= 0;
    // pages outside the pool read page 0's summaries (their score is -inf)
    const uint16_t* meta = p.meta_pool + (size_t)(load ? phys : 0) * 2 * D + g * CH;
    uint4 mn[C4], mx[C4];
#pragma unroll
    for (int i = 0; i < C4; ++i) {
      mn[i] = reinterpret_cast<const uint4*>(meta)[i];
      mx[i] = reinterpret_cast<const uint4*>(meta + D)[i];
    }
    const float best = page_bound<D, G>(qp, qn, mn, mx);
    if (valid && g == 0) p.scores[(size_t)unit * p.scores_stride + b] = load ? best * p.scale : -INFINITY;
  }
}

__global__ __launch_bounds__(256) void quest_topk_kernel(const QuestParams p) {
  constexpr int NT = 256;
  __shared__ unsigned hist[256];
  __shared__ int scan_scratch[NT / kWave + 1];
  __shared__ int bcast[4];
  const int tid = threadIdx.x;
  const int unit = blockIdx.x;
  const int L = p.lengths[unit];
  int32_t* out = p.sel + (size_t)unit * p.top_k;
  if (!unit_length_ok(p, L)) {
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    for (int i = tid; i < p.top_k; i += NT) out[i] = -1;
    return;
  }
  const int n = L / kPage;
  if (n <= p.top_k) {
    for (int i = tid; i < p.top_k; i += NT) out[i] = i < n ? i : -1;
    return;
  }
  const float* sc = p.scores + (size_t)unit * p.scores_stride;
  auto key_of = [&](int b) { return float_key(sc[b]); };
  uint32_t prefix, mask;
  int k_rest;
  radix_select_top<NT, uint32_t>(n, p.top_k, key_of, [](int) { return true; }, &prefix, &mask,
                                 &k_rest, hist, scan_scratch, bcast);
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
    if (take) out[out_base + rank] = b;
    eq_base += eq_total;
    out_base += take_total;
  }
}

constexpr int kFusedThreads = 1024;
constexpr int kFusedMaxPages = 8192;
constexpr int kFusedMinUnits = 256;  // one work-group per unit fills the compute units

template <int D, int G>
__global__ __launch_bounds__(kFusedThreads) void quest_select_fused_kernel(const QuestParams p) {
  constexpr int NT = kFusedThreads;
  __shared__ int lds_bt[kFusedMaxPages];
  __shared__ float lds_sc[kFusedMaxPages];
  __shared__ unsigned hist[256];
  __shared__ unsigned hist2[256];
  __shared__ int bcast[4];
  const int tid = threadIdx.x;
  const int unit = blockIdx.x;
  const int L = p.lengths[unit];
  int32_t* out = p.sel + (size_t)unit * p.top_k;
  if (!unit_length_ok(p, L) || L / kPage > kFusedMaxPages) {
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    for (int i = tid; i < p.top_k; i += NT) out[i] = -1;
    return;
  }
  const int n = L / kPage;
  int bad = 0;
  for (int i = tid; i < n; i += NT) {
    int ph = p.block_table[(size_t)unit * p.max_pages + i];
    if (ph < 0 || (int64_t)ph >= p.num_pages) {
      bad = 1;
      ph = -1;
    }
    lds_bt[i] = ph;
  }
  if (bad) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
  if (tid < 256) {
    hist[tid] = 0;
    hist2[tid] = 0;
  }
  __syncthreads();
  const int req = unit / p.hkv, kvh = unit - req * p.hkv;
  unit_bounds<NT, D, G>(p.meta_pool, p.q + ((size_t)req * p.hkv * G + (size_t)kvh * G) * D, p.scale, n, lds_bt,
                        lds_sc, p.write_scores ? p.scores + (size_t)unit * p.scores_stride : nullptr, hist, hist2);
  __syncthreads();
  unit_topk<NT>(n, p.top_k, lds_sc, [&](int r, int b) { out[r] = b; }, hist, hist2, bcast, true);
}

}  // namespace se

using namespace se;

size_t se_quest_workspace_bytes(int32_t num_units, int32_t max_pages) {
  if (num_units <= 0 || max_pages <= 0) return 0;
  return align_up((size_t)num_units * max_pages * 4, 256);
}

extern "C" se_status se_quest_summarize(const se_kv_view* kv, int32_t max_len, int32_t* dev_err,
                                        hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->kv_pool == nullptr || kv->meta_pool == nullptr || dev_err == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if (max_len < 1) return SE_ERR_INVALID_ARGUMENT;
  QuestParams prm = {};
  prm.kv = static_cast<const uint16_t*>(kv->kv_pool);
  prm.meta_pool = static_cast<uint16_t*>(kv->meta_pool);
  prm.block_table = kv->block_table;
  prm.lengths = kv->lengths;
  prm.num_pages = kv->num_pages;
  prm.hkv = kv->num_kv_heads;
  prm.max_pages = kv->max_pages;
  prm.max_len = max_len;
  prm.dev_err = dev_err;
  int64_t ml = max_len;
  if (ml > (int64_t)kv->max_pages * kPage) ml = (int64_t)kv->max_pages * kPage;
  prm.blocks_per_unit = (int)ceil_div(ceil_div(ml, kPage), 4);
  const int64_t grid = (int64_t)kv->num_units * prm.blocks_per_unit;
  if (grid > INT32_MAX) return SE_ERR_UNSUPPORTED;
  if (kv->head_dim == 128)
    hipLaunchKernelGGL((quest_summarize_kernel<128>), dim3((int)grid), dim3(256), 0, stream, prm);
  else
    hipLaunchKernelGGL((quest_summarize_kernel<64>), dim3((int)grid), dim3(256), 0, stream, prm);
  return launch_status();
}

extern "C" se_status se_quest_select(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                                     float scale, int32_t top_k, int32_t max_len, uint32_t flags,
                                     int32_t* sel_pages, float* page_scores, int32_t scores_stride,
                                     void* ws, size_t ws_bytes, int32_t* dev_err,
                                     hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if ((flags & ~SE_QUEST_SCORES_GIVEN) != 0) return SE_ERR_INVALID_ARGUMENT;
  const bool given = (flags & SE_QUEST_SCORES_GIVEN) != 0;
  if (sel_pages == nullptr || dev_err == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (top_k < 1 || top_k > 4096 || max_len < 1) return SE_ERR_INVALID_ARGUMENT;
  if (given && page_scores == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (page_scores != nullptr && scores_stride < kv->max_pages) return SE_ERR_INVALID_ARGUMENT;
  if (!given) {
    if (q == nullptr || kv->meta_pool == nullptr) return SE_ERR_INVALID_ARGUMENT;
    if (q_per_kv != 1 && q_per_kv != 2 && q_per_kv != 4 && q_per_kv != 8) return SE_ERR_UNSUPPORTED;
    if (!(scale > 0.f)) return SE_ERR_INVALID_ARGUMENT;
  }
  QuestParams prm = {};
  prm.kv = static_cast<const uint16_t*>(kv->kv_pool);
  prm.meta_pool = static_cast<uint16_t*>(kv->meta_pool);
  prm.block_table = kv->block_table;
  prm.lengths = kv->lengths;
  prm.num_pages = kv->num_pages;
  prm.hkv = kv->num_kv_heads;
  prm.max_pages = kv->max_pages;
  prm.max_len = max_len;
  prm.q = static_cast<const uint16_t*>(q);
  prm.scale = scale;
  prm.top_k = top_k;
  prm.sel = sel_pages;
  prm.dev_err = dev_err;
  if (page_scores != nullptr) {
    prm.scores = page_scores;
    prm.scores_stride = scores_stride;
  } else {
    if (ws == nullptr || ws_bytes < se_quest_workspace_bytes(kv->num_units, kv->max_pages))
      return SE_ERR_WORKSPACE;
    prm.scores = static_cast<float*>(ws);
    prm.scores_stride = kv->max_pages;
  }
  if (!given) {
    int64_t ml = max_len;
    if (ml > (int64_t)kv->max_pages * kPage) ml = (int64_t)kv->max_pages * kPage;
    if (kv->num_units >= kFusedMinUnits && ml / kPage <= kFusedMaxPages) {
      prm.write_scores = page_scores != nullptr ? 1 : 0;
      const int D = kv->head_dim;
      const dim3 grid(kv->num_units), block(kFusedThreads);
      if (D == 128) {
        if (q_per_kv == 8) hipLaunchKernelGGL((quest_select_fused_kernel<128, 8>), grid, block, 0, stream, prm);
        else if (q_per_kv == 4) hipLaunchKernelGGL((quest_select_fused_kernel<128, 4>), grid, block, 0, stream, prm);
        else if (q_per_kv == 2) hipLaunchKernelGGL((quest_select_fused_kernel<128, 2>), grid, block, 0, stream, prm);
        else hipLaunchKernelGGL((quest_select_fused_kernel<128, 1>), grid, block, 0, stream, prm);
      } else {
        if (q_per_kv == 8) hipLaunchKernelGGL((quest_select_fused_kernel<64, 8>), grid, block, 0, stream, prm);
        else if (q_per_kv == 4) hipLaunchKernelGGL((quest_select_fused_kernel<64, 4>), grid, block, 0, stream, prm);
        else if (q_per_kv == 2) hipLaunchKernelGGL((quest_select_fused_kernel<64, 2>), grid, block, 0, stream, prm);
        else hipLaunchKernelGGL((quest_select_fused_kernel<64, 1>), grid, block, 0, stream, prm);
      }
      return launch_status();
    }
    prm.blocks_per_unit = (int)ceil_div(ml / kPage > 0 ? ml / kPage : 1, kBoundPagesPerGroup);
    const int64_t grid = (int64_t)kv->num_units * prm.blocks_per_unit;
    if (grid > INT32_MAX) return SE_ERR_UNSUPPORTED;
    const int D = kv->head_dim;
    if (D == 128) {
      if (q_per_kv == 8) hipLaunchKernelGGL((quest_bound_kernel<128, 8>), dim3((int)grid), dim3(256), 0, stream, prm);
      else if (q_per_kv == 4) hipLaunchKernelGGL((quest_bound_kernel<128, 4>), dim3((int)grid), dim3(256), 0, stream, prm);
      else if (q_per_kv == 2) hipLaunchKernelGGL((quest_bound_kernel<128, 2>), dim3((int)grid), dim3(256), 0, stream, prm);
      else hipLaunchKernelGGL((quest_bound_kernel<128, 1>), dim3((int)grid), dim3(256), 0, stream, prm);
    } else {
      if (q_per_kv == 8) hipLaunchKernelGGL((quest_bound_kernel<64, 8>), dim3((int)grid), dim3(256), 0, stream, prm);
      else if (q_per_kv == 4) hipLaunchKernelGGL((quest_bound_kernel<64, 4>), dim3((int)grid), dim3(256), 0, stream, prm);
      else if (q_per_kv == 2) hipLaunchKernelGGL((quest_bound_kernel<64, 2>), dim3((int)grid), dim3(256), 0, stream, prm);
      else hipLaunchKernelGGL((quest_bound_kernel<64, 1>), dim3((int)grid), dim3(256), 0, stream, prm);
    }
    st = launch_status();
    if (st != SE_OK) return st;
  }
  hipLaunchKernelGGL(quest_topk_kernel, dim3(kv->num_units), dim3(256), 0, stream, prm);
  return launch_status();
}
