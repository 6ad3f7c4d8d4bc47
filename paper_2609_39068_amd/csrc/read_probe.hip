// se_probe_read_pages: the plain read rate of a page-gather pattern, measured
// with the decode stream's own loads.  It is the ceiling an HBM-bound kernel
// reading the same pages can reach, and the figure the decode kernels' rates
// are compared with.  A measurement aid: no step of the method runs here.
//
// Every wavefront reads whole 8 KiB pages (list entries wave, wave + W, ...,
// W the wavefronts of the grid), two pages per iteration with all their
// 16-byte nontemporal loads in flight (16 per lane), and XOR-folds the words
// into one value per lane, stored at the end so the loads are not removed.
#include "se_common.h"

namespace se {

constexpr int kProbeThreads = 512;
constexpr int kProbePageBytes = 8192;

typedef uint32_t probe_u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kProbeThreads) void probe_read_kernel(const char* pool, int64_t pool_pages,
                                                                   const int32_t* pages, int64_t n_pages,
                                                                   uint32_t* sink) {
  constexpr int CH = kProbePageBytes / (kWave * 16);  // 16-byte loads per lane per page
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = (int64_t)blockIdx.x * (kProbeThreads / kWave) + (threadIdx.x / kWave);
  const int64_t nw = (int64_t)gridDim.x * (kProbeThreads / kWave);
  auto page_at = [&](int64_t i) -> const char* {
    int ph = pages[i < n_pages ? i : n_pages - 1];
    ph = __builtin_amdgcn_readfirstlane(ph);
    if (ph < 0 || (int64_t)ph >= pool_pages) ph = 0;
    return pool + (size_t)ph * kProbePageBytes + lane * 16;
  };
  uint32_t acc = 0;
  for (int64_t i = wave; i < n_pages; i += 2 * nw) {
    const char* a = page_at(i);
    const char* b = page_at(i + nw);  // past the end: the last page again, not folded
    probe_u32x4 va[CH], vb[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) va[c] = __builtin_nontemporal_load(reinterpret_cast<const probe_u32x4*>(a + c * 1024));
#pragma unroll
    for (int c = 0; c < CH; ++c) vb[c] = __builtin_nontemporal_load(reinterpret_cast<const probe_u32x4*>(b + c * 1024));
    const bool use_b = i + nw < n_pages;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      acc ^= va[c].x ^ va[c].y ^ va[c].z ^ va[c].w;
      if (use_b) acc ^= vb[c].x ^ vb[c].y ^ vb[c].z ^ vb[c].w;
    }
  }
  sink[(size_t)blockIdx.x * kProbeThreads + threadIdx.x] = acc;
}

}  // namespace se

using namespace se;

extern "C" se_status se_probe_read_pages(const void* pool, int64_t pool_pages, const int32_t* pages,
                                         int64_t n_pages, int32_t page_bytes, int32_t grid, uint32_t* sink,
                                         hipStream_t stream) {
  if (pool == nullptr || pages == nullptr || sink == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (page_bytes != kProbePageBytes || grid < 1 || n_pages < 1 || pool_pages < 1) return SE_ERR_INVALID_ARGUMENT;
  hipLaunchKernelGGL(probe_read_kernel, dim3(grid), dim3(kProbeThreads), 0, stream,
                     static_cast<const char*>(pool), pool_pages, pages, n_pages, sink);
  return launch_status();
}
