// se_accumulate_scores (the unfused H2O score update) and the small C-ABI
// utilities: workspace sizes, the device error word, status names, version.
#include "se_common.h"

namespace se {

struct AccumParams {
  float* score_pool;
  const int32_t* block_table;
  const int32_t* lengths;
  int64_t num_pages;
  int32_t hkv;
  int32_t max_pages;
  int32_t max_len;
  int32_t G;
  const float* logits;
  int32_t logits_stride;
  const float* lse;
  int32_t blocks_per_unit;
  int32_t* dev_err;
};

// eq. background-h2o-score: score(j) += sum over the group of exp(z_a(j) - lse_a).
__global__ __launch_bounds__(256) void accumulate_scores_kernel(const AccumParams p) {
  const int unit = blockIdx.x / p.blocks_per_unit;
  const int s = (blockIdx.x - unit * p.blocks_per_unit) * 256 + threadIdx.x;
  const int L = p.lengths[unit];
  if (L < 0 || L > p.max_len || L > p.max_pages * kPage) {
    if (s == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return;
  }
  if (s >= L) return;
  const int phys = p.block_table[(size_t)unit * p.max_pages + s / kPage];
  if (phys < 0 || (int64_t)phys >= p.num_pages) {
    if ((s & (kPage - 1)) == 0) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
    return;
  }
  const int req = unit / p.hkv;
  const int kvh = unit - req * p.hkv;
  float a = 0.f;
  for (int h = 0; h < p.G; ++h) {
    const float z = p.logits[((size_t)unit * p.G + h) * p.logits_stride + s];
    const float l = p.lse[(size_t)req * p.hkv * p.G + kvh * p.G + h];
    a += __expf(z - l);
  }
  p.score_pool[(size_t)phys * kPage + (s & (kPage - 1))] += a;
}

}  // namespace se

using namespace se;

extern "C" se_status se_accumulate_scores(const se_kv_view* kv, int32_t q_per_kv,
                                          const float* logits, int32_t logits_stride,
                                          const float* lse, int32_t max_len, int32_t* dev_err,
                                          hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->score_pool == nullptr || logits == nullptr || lse == nullptr || dev_err == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if (q_per_kv < 1 || q_per_kv > 8) return SE_ERR_UNSUPPORTED;
  if (max_len < 1 || logits_stride < max_len) return SE_ERR_INVALID_ARGUMENT;
  AccumParams prm;
  prm.score_pool = kv->score_pool;
  prm.block_table = kv->block_table;
  prm.lengths = kv->lengths;
  prm.num_pages = kv->num_pages;
  prm.hkv = kv->num_kv_heads;
  prm.max_pages = kv->max_pages;
  prm.max_len = max_len;
  prm.G = q_per_kv;
  prm.logits = logits;
  prm.logits_stride = logits_stride;
  prm.lse = lse;
  prm.blocks_per_unit = (int)ceil_div(max_len, 256);
  prm.dev_err = dev_err;
  const int64_t grid = (int64_t)kv->num_units * prm.blocks_per_unit;
  if (grid > INT32_MAX) return SE_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(accumulate_scores_kernel, dim3((int)grid), dim3(256), 0, stream, prm);
  return launch_status();
}

extern "C" size_t se_workspace_bytes(int32_t op, int32_t num_units, int32_t max_len,
                                     int32_t max_pages, int32_t q_per_kv, int32_t head_dim,
                                     int32_t top_k) {
  switch (op) {
    case SE_OP_DECODE_ATTEND:
      return se_attend_workspace_bytes(num_units, max_len, max_pages, q_per_kv, head_dim,
                                       top_k > 0 ? top_k : 0);
    case SE_OP_QUEST_SELECT:
      return se_quest_workspace_bytes(num_units, max_pages);
    case SE_OP_QUEST_STEP:
      return se_quest_step_workspace_bytes(num_units, max_len, max_pages, q_per_kv, head_dim, top_k);
    case SE_OP_SNAPKV:
      return se_snapkv_workspace_bytes(num_units, max_len, q_per_kv, top_k);
    case SE_OP_OMNIKV_SELECT:
      return se_omnikv_workspace_bytes(num_units, max_len);
    case SE_OP_H2O_PREFILL:
      return se_h2o_prefill_workspace_bytes(num_units, max_len, q_per_kv, top_k);
    default:
      return 0;
  }
}

extern "C" se_status se_read_device_errors(int32_t* dev_err, int32_t* host_out,
                                           hipStream_t stream) {
  if (dev_err == nullptr || host_out == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (hipMemcpyAsync(host_out, dev_err, sizeof(int32_t), hipMemcpyDeviceToHost, stream) !=
      hipSuccess)
    return SE_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return SE_ERR_HIP;
  if (hipMemsetAsync(dev_err, 0, sizeof(int32_t), stream) != hipSuccess) return SE_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return SE_ERR_HIP;
  return SE_OK;
}

extern "C" const char* se_status_string(se_status status) {
  switch (status) {
    case SE_OK: return "SE_OK";
    case SE_ERR_INVALID_ARGUMENT: return "SE_ERR_INVALID_ARGUMENT";
    case SE_ERR_UNSUPPORTED: return "SE_ERR_UNSUPPORTED";
    case SE_ERR_WORKSPACE: return "SE_ERR_WORKSPACE";
    case SE_ERR_HIP: return "SE_ERR_HIP";
  }
  return "SE_UNKNOWN_STATUS";
}

extern "C" int32_t se_version(void) { return 100; }
