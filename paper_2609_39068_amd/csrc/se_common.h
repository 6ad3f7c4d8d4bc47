// Shared device and host helpers of the sparse-engine HIP library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sparse_engine.h"

namespace se {

constexpr int kPage = 16;          // slots per page
constexpr int kWave = 64;          // CDNA wavefront width
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// ---------------------------------------------------------------- host side

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Checks the fields of a view that every operation relies on.
inline se_status check_view(const se_kv_view* kv) {
  if (kv == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (kv->num_units <= 0 || kv->num_kv_heads <= 0 || kv->max_pages <= 0 || kv->num_pages <= 0)
    return SE_ERR_INVALID_ARGUMENT;
  if (kv->num_units % kv->num_kv_heads != 0) return SE_ERR_INVALID_ARGUMENT;
  if (kv->block_table == nullptr || kv->lengths == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (kv->page_size != kPage) return SE_ERR_UNSUPPORTED;
  if (kv->head_dim != 64 && kv->head_dim != 128) return SE_ERR_UNSUPPORTED;
  if (kv->num_pages > (int64_t)INT32_MAX) return SE_ERR_UNSUPPORTED;
  return SE_OK;
}

inline se_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? SE_OK : SE_ERR_HIP;
}

// Split-K shape of se_decode_attend: how many work-groups share one unit and
// how many visited pages each of them streams.  A pure function of the sizes,
// so the workspace query and the launch agree.
struct SplitShape {
  int n_visit;   // pages visited per unit at most
  int n_split;   // work-groups per unit
  int pps;       // pages per work-group
};

// resident: work-groups that fit the chip at once (512: two 8-wavefront
// work-groups on each of 256 compute units; 256: one 16-wavefront one).
inline SplitShape split_shape(int num_units, int n_visit, int resident = 512) {
  const int min_pages = 16;          // at least two pages per wavefront
  const int max_group_pages = 1024;  // the page table a work-group stages in LDS
  int splits = (int)ceil_div(resident, num_units);
  int by_size = (int)ceil_div(n_visit, min_pages);
  if (splits > by_size) splits = by_size;
  if (splits < 1) splits = 1;
  if (splits < ceil_div(n_visit, max_group_pages)) splits = (int)ceil_div(n_visit, max_group_pages);
  int pps = (int)ceil_div(n_visit, splits);
  splits = (int)ceil_div(n_visit, pps);
  return SplitShape{n_visit, splits, pps};
}

// ---------------------------------------------------------------- device side

__device__ __forceinline__ float bf16lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }
__device__ __forceinline__ float bf16f(uint16_t x) { return __uint_as_float(((uint32_t)x) << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// acc + a.lo*b.lo + a.hi*b.hi on packed bf16 pairs (v_dot2c_f32_bf16).
__device__ __forceinline__ float dot2bf16(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), acc, false);
}

// DPP quad permutations: lane i of each group of four reads lane perm[i].
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]

// Sum over the four lanes of a quad, result in all four.
__device__ __forceinline__ float quad_sum(float v) {
  v += dpp_f<kQuadXor1>(v);
  v += dpp_f<kQuadXor2>(v);
  return v;
}

__device__ __forceinline__ float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, kWave); }

__device__ __forceinline__ float wave_max(float v) {
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, shfl_xor_f(v, m));
  return v;
}

__device__ __forceinline__ int ceil_div_dev(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ void set_error(int32_t* dev_err, uint32_t bit) {
  atomicOr(dev_err, (int32_t)bit);
}

// Order-preserving map of a float to uint32 (larger float -> larger key);
// -0 is folded onto +0 so that equal values compare equal.
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t b = __float_as_uint(f + 0.0f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Block-wide exclusive scan of one int per thread (blockDim.x == NT, NT % 64 == 0).
// `scratch` holds NT/64 + 1 ints of LDS.  Returns the exclusive prefix; *total the sum.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int* scratch, int* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  int x = v;
  for (int o = 1; o < kWave; o <<= 1) {
    int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) scratch[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < NT / kWave; ++w) {
      int t = scratch[w];
      scratch[w] = run;
      run += t;
    }
    scratch[NT / kWave] = run;
  }
  __syncthreads();
  int res = x - v + scratch[wave];
  *total = scratch[NT / kWave];
  __syncthreads();
  return res;
}

// Block-wide reductions (blockDim.x == NT).  `scratch` holds NT/64 values.
template <int NT, typename T, typename Op>
__device__ __forceinline__ T block_reduce(T v, T* scratch, Op op) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  for (int o = 32; o >= 1; o >>= 1) v = op(v, __shfl_xor(v, o, kWave));
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  T r = scratch[0];
  for (int w = 1; w < NT / kWave; ++w) r = op(r, scratch[w]);
  __syncthreads();
  return r;
}

// Radix selection of the k largest keys among the items for which cand(i) holds
// (blockDim.x == NT, NT >= 256; 8-bit digits, one histogram bin per thread).  After the call, an item is among the k largest
// iff (key & *mask) > *prefix, or (key & *mask) == *prefix and it is one of the
// first *k_rest such items in index order.  Needs k >= 1 and at least k candidates.
template <int NT, typename KeyT, typename KeyFn, typename CandFn>
__device__ void radix_select_top(int n, int k, KeyFn key_of, CandFn cand, KeyT* prefix_out,
                                 KeyT* mask_out, int* k_rest_out, unsigned* hist, int* scan_scratch,
                                 int* bcast) {
  static_assert(NT >= 256 && NT % kWave == 0, "threads 0..255 own one bin each");
  KeyT prefix = 0, mask = 0;
  const int tid = threadIdx.x;
  for (int shift = (int)sizeof(KeyT) * 8 - 8; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int i = tid; i < n; i += NT) {
      if (!cand(i)) continue;
      const KeyT key = key_of(i);
      if ((key & mask) == prefix) atomicAdd(&hist[(unsigned)(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    const int v = tid < 256 ? (int)hist[255 - tid] : 0;  // thread t counts digit 255 - t
    int total;
    const int excl = block_exclusive_scan<NT>(v, scan_scratch, &total);
    if (v > 0 && excl < k && excl + v >= k) {
      bcast[0] = 255 - tid;
      bcast[1] = excl;
      bcast[2] = v;
    }
    __syncthreads();
    const int d = bcast[0];
    k -= bcast[1];
    const int cnt = bcast[2];
    __syncthreads();
    prefix |= (KeyT)d << shift;
    mask |= (KeyT)0xFF << shift;
    if (cnt == k) break;
  }
  *prefix_out = prefix;
  *mask_out = mask;
  *k_rest_out = k;
}

}  // namespace se

// Workspace sizes of the operations that need one (defined next to their kernels).
size_t se_attend_workspace_bytes(int32_t num_units, int32_t max_len, int32_t max_pages,
                                 int32_t q_per_kv, int32_t head_dim, int32_t top_k);
size_t se_quest_workspace_bytes(int32_t num_units, int32_t max_pages);
size_t se_snapkv_workspace_bytes(int32_t num_units, int32_t max_len, int32_t q_per_kv, int32_t window);
size_t se_omnikv_workspace_bytes(int32_t num_req, int32_t max_len);
size_t se_h2o_prefill_workspace_bytes(int32_t num_units, int32_t max_len, int32_t q_per_kv, int32_t window);
size_t se_quest_step_workspace_bytes(int32_t num_units, int32_t max_len, int32_t max_pages, int32_t q_per_kv,
                                     int32_t head_dim, int32_t top_k);


