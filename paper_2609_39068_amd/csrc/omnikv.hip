// OmniKV cross-layer selection (Appendix A.3, "OmniKV: Selection Reuse across
// Layers", eqs. background-omnikv-selection and background-omnikv-reuse):
//   se_omnikv_select  at an observation layer, from the logits se_decode_attend
//                     wrote for every resident slot: s(j) = max over the
//                     request's query heads of z_j, then TopK_b of s per request;
//   se_attend_slots   at a sparse layer: append the decode token, then each
//                     KV head's group attends over the selected slots of its
//                     own cache.
//
// Selection: omnikv_score_kernel takes the maximum over the request's Hq
// logit rows (contiguous in the logits layout) for a chunk of slots, coalesced,
// into the workspace; omnikv_topk_kernel (one 1024-thread work-group per
// request) copies the request's scores to LDS when they fit (eight loads in
// flight per thread), finds the b-th largest key by an 8-bit radix selection
// over order-preserving keys (ties: lower slot; the histogram replicated over
// eight LDS copies, so that lanes sharing a digit update different words), and
// writes the selected slots in increasing order: every thread owns a
// contiguous run of slots, so two block scans (of the tied count and of the
// selected count) give each thread its output offset.
//
// Slot attention: one 512-thread work-group per unit.  The selected slots are
// translated once into kv-pool row indices in LDS (the appended token's row is
// read from k_new / v_new instead, so no wavefront reads a row another one
// wrote).  Each wavefront takes a contiguous share of the rows, eight rows per
// pass: for QK, 8 lanes share a key row (D/8 columns each, 16-byte loads) and
// reduce their bf16-pair dot products over the 8 lanes; the online softmax
// keeps one maximum per head; the pass's weights are broadcast through LDS and
// every lane accumulates its own D/64 value columns of the 8 rows (one
// coalesced row per load instruction).  The next pass's key and value loads
// are issued before the current pass is reduced.  Wavefronts combine in LDS.
#include "quest_core.h"

namespace se {

constexpr int kOmniScoreThreads = 256;
constexpr int kOmniScoreSlots = 4;                      // slots per thread per block
constexpr int kOmniTopkThreads = 1024;
constexpr int kOmniLdsScores = 32768 + 4096;            // scores kept in LDS (144 KB)
constexpr int kOmniHistCopies = 8;                      // radix histogram copies (8 KB of LDS)
constexpr int kOmniRowBatch = 8;                        // logit rows in flight per thread
constexpr int kGatherThreads = 512;       // two work-groups per compute unit
constexpr int kGatherThreadsWide = 1024;  // at most one work-group per compute unit: twice the rows in flight
constexpr int kGatherMaxSel = 8192;                     // selected slots per request
constexpr uint32_t kNewRow = 0xFFFFFFFFu;               // the appended token (read from k_new / v_new)

struct OmniSelectParams {
  const float* logits;   // [num_units][G][stride]
  int32_t stride;
  const int32_t* lengths;
  int32_t num_req;
  int32_t num_kv_heads;
  int32_t q_per_kv;
  int32_t budget;
  int32_t max_len;
  int32_t ws_stride;
  int32_t vec4;          // logits rows 16-byte aligned: four slots per load
  float* scores;         // workspace [num_req][ws_stride]
  int32_t* sel;          // [num_req][budget]
  int32_t* dev_err;
};

// radix_select_top (se_common.h) with the histogram replicated COPIES times (copy = lane
// mod COPIES, copies 257 words apart, so in different banks): lanes that share
// a digit -- most of them in the first passes over scores of similar
// magnitude -- then update different LDS words instead of serialising on one.
// `hist` holds COPIES * 257 words.
template <int NT, int COPIES, typename KeyT, typename KeyFn, typename CandFn>
__device__ void radix_select_top_rep(int n, int k, KeyFn key_of, CandFn cand, KeyT* prefix_out, KeyT* mask_out,
                                     int* k_rest_out, unsigned* hist, int* bcast) {
  static_assert(NT % kWave == 0, "whole wavefronts");
  constexpr int kStride = 257;
  KeyT prefix = 0, mask = 0;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  unsigned* const my_hist = hist + (tid % COPIES) * kStride;
  for (int i = tid; i < COPIES * kStride; i += NT) hist[i] = 0;
  __syncthreads();
  // two barriers a pass: the counts are in; then wavefront 0 alone sums the
  // copies (clearing them for the next pass), scans the 256 digits and
  // broadcasts the threshold digit
  for (int shift = (int)sizeof(KeyT) * 8 - 8; shift >= 0; shift -= 8) {
    for (int i = tid; i < n; i += NT) {
      if (!cand(i)) continue;
      const KeyT key = key_of(i);
      if ((key & mask) == prefix) atomicAdd(&my_hist[(unsigned)(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < kWave) {
      // lane l holds digits 255-4l .. 252-4l (descending); inclusive prefix over lanes
      int c[4], s4 = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int v = 0;
#pragma unroll
        for (int cp = 0; cp < COPIES; ++cp) {
          unsigned* const w = hist + cp * kStride + 255 - 4 * lane - j;
          v += (int)*w;
          *w = 0u;
        }
        c[j] = v;
        s4 += v;
      }
      int incl = s4;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
      }
      int run = incl - s4;  // candidates in higher digits than this lane's first
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (c[j] > 0 && run < k && run + c[j] >= k) {
          bcast[0] = 255 - 4 * lane - j;
          bcast[1] = run;
          bcast[2] = c[j];
        }
        run += c[j];
      }
    }
    __syncthreads();
    const int d = bcast[0];
    k -= bcast[1];
    const int cnt = bcast[2];
    prefix |= (KeyT)d << shift;
    mask |= (KeyT)0xFF << shift;
    if (cnt == k) break;
  }
  *prefix_out = prefix;
  *mask_out = mask;
  *k_rest_out = k;
}

// s(j) = max over the request's Hkv * G logit rows, for slots j < L of the
// request's first unit.  With aligned rows a thread takes four consecutive
// slots per 16-byte load and keeps eight rows' loads in flight (slots past L up
// to the next multiple of four get scores nobody reads: they stay inside the
// rows, whose stride is a multiple of four at least max_len).
__global__ __launch_bounds__(kOmniScoreThreads) void omnikv_score_kernel(const OmniSelectParams p) {
  const int req = blockIdx.y;
  const int L = p.lengths[(size_t)req * p.num_kv_heads];
  const int rows = p.num_kv_heads * p.q_per_kv;
  const float* lg = p.logits + (size_t)req * rows * p.stride;
  if (L < 0 || L > p.max_len) return;  // reported by the selection kernel
  if (p.vec4) {
    const int j0 = (blockIdx.x * kOmniScoreThreads + threadIdx.x) * kOmniScoreSlots;
    if (j0 >= L) return;
    float4 m = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    int r = 0;
    for (; r + kOmniRowBatch <= rows; r += kOmniRowBatch) {
      float4 v[kOmniRowBatch];
#pragma unroll
      for (int k = 0; k < kOmniRowBatch; ++k) v[k] = *reinterpret_cast<const float4*>(lg + (size_t)(r + k) * p.stride + j0);
#pragma unroll
      for (int k = 0; k < kOmniRowBatch; ++k) {
        m.x = fmaxf(m.x, v[k].x);
        m.y = fmaxf(m.y, v[k].y);
        m.z = fmaxf(m.z, v[k].z);
        m.w = fmaxf(m.w, v[k].w);
      }
    }
    for (; r < rows; ++r) {
      const float4 v = *reinterpret_cast<const float4*>(lg + (size_t)r * p.stride + j0);
      m.x = fmaxf(m.x, v.x);
      m.y = fmaxf(m.y, v.y);
      m.z = fmaxf(m.z, v.z);
      m.w = fmaxf(m.w, v.w);
    }
    *reinterpret_cast<float4*>(p.scores + (size_t)req * p.ws_stride + j0) = m;
    return;
  }
  const int base = blockIdx.x * kOmniScoreThreads * kOmniScoreSlots + threadIdx.x;
#pragma unroll
  for (int k = 0; k < kOmniScoreSlots; ++k) {
    const int j = base + k * kOmniScoreThreads;
    if (j >= L) break;
    float s = -INFINITY;
    for (int r = 0; r < rows; ++r) s = fmaxf(s, lg[(size_t)r * p.stride + j]);
    p.scores[(size_t)req * p.ws_stride + j] = s;
  }
}

__global__ __launch_bounds__(kOmniTopkThreads) void omnikv_topk_kernel(const OmniSelectParams p) {
  __shared__ __attribute__((aligned(16))) float s_sc[kOmniLdsScores];
  __shared__ unsigned s_hist[kOmniHistCopies * 257];
  __shared__ int s_scan[kOmniTopkThreads / kWave + 1];
  __shared__ int s_bcast[4];
  const int req = blockIdx.x;
  const int tid = threadIdx.x;
  int32_t* out = p.sel + (size_t)req * p.budget;
  const int L = p.lengths[(size_t)req * p.num_kv_heads];
  int bad = (L < 0 || L > p.max_len) ? 1 : 0;
  for (int h = 1; h < p.num_kv_heads; ++h) bad |= (p.lengths[(size_t)req * p.num_kv_heads + h] != L);
  if (bad) {  // every unit of a request keeps the whole history: the lengths agree
    for (int i = tid; i < p.budget; i += kOmniTopkThreads) out[i] = -1;
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return;
  }
  const int b = p.budget;
  if (L <= b) {
    for (int i = tid; i < b; i += kOmniTopkThreads) out[i] = i < L ? i : -1;
    return;
  }
  const float* gsc = p.scores + (size_t)req * p.ws_stride;
  const float* sc = gsc;
  if (L <= kOmniLdsScores) {
    // eight loads in flight per thread (16-byte ones when the rows are aligned);
    // the loads are unconditional (an index past the end re-reads the last
    // element, which is not stored), so the values stay in registers and no
    // load waits for the one before it
    constexpr int NB = 8;
    int done = 0;
    if (p.vec4) {
      const int n4 = L / 4;
      for (int i = tid; i < n4; i += kOmniTopkThreads * NB) {
        float4 v[NB];
#pragma unroll
        for (int k = 0; k < NB; ++k)
          v[k] = reinterpret_cast<const float4*>(gsc)[min(i + k * kOmniTopkThreads, n4 - 1)];
#pragma unroll
        for (int k = 0; k < NB; ++k) {
          const int x = i + k * kOmniTopkThreads;
          if (x < n4) reinterpret_cast<float4*>(s_sc)[x] = v[k];
        }
      }
      done = 4 * n4;
    }
    for (int i = done + tid; i < L; i += kOmniTopkThreads * NB) {
      float v[NB];
#pragma unroll
      for (int k = 0; k < NB; ++k) v[k] = gsc[min(i + k * kOmniTopkThreads, L - 1)];
#pragma unroll
      for (int k = 0; k < NB; ++k) {
        const int x = i + k * kOmniTopkThreads;
        if (x < L) s_sc[x] = v[k];
      }
    }
    __syncthreads();
    sc = s_sc;
  }
  uint32_t prefix, mask;
  int k_rest;
  radix_select_top_rep<kOmniTopkThreads, kOmniHistCopies, uint32_t>(
      L, b, [&](int i) { return float_key(sc[i]); }, [](int) { return true; }, &prefix, &mask, &k_rest, s_hist,
      s_bcast);
  // thread t owns slots [t*run, (t+1)*run): count the threshold ties, rank them
  // in slot order, then place the selected slots
  const int run = ceil_div_dev(L, kOmniTopkThreads);
  const int lo = min(L, tid * run), hi = min(L, lo + run);
  int tot;
  if (run <= 64) {
    // one pass over the run builds two masks (bit j: slot lo + j above the
    // threshold, equal to it), read in an order rotated by the thread so that
    // a wavefront's lanes read different banks; the counts, the ties taken
    // (the first k_rest - eq_before of the block's ties, in slot order) and
    // the output offsets then come from the masks alone
    const int n = hi - lo;
    const int rot = (tid >> 1) % run;
    uint64_t gt = 0, eq = 0;
    for (int j = 0; j < run; ++j) {
      const int jj = j + rot < run ? j + rot : j + rot - run;
      if (jj < n) {
        const uint32_t km = float_key(sc[lo + jj]) & mask;
        gt |= (uint64_t)(km > prefix) << jj;
        eq |= (uint64_t)(km == prefix) << jj;
      }
    }
    const int n_eq = __popcll(eq);
    const int eq_before = block_exclusive_scan<kOmniTopkThreads>(n_eq, s_scan, &tot);
    uint64_t selm = gt;
    for (int t = min(max(k_rest - eq_before, 0), n_eq); t > 0; --t) {
      const uint64_t low = eq & (~eq + 1);  // the lowest remaining tie
      selm |= low;
      eq ^= low;
    }
    int o = block_exclusive_scan<kOmniTopkThreads>(__popcll(selm), s_scan, &tot);
    while (selm != 0) {
      out[o++] = lo + __builtin_ctzll(selm);
      selm &= selm - 1;
    }
    return;
  }
  int n_eq = 0;
  for (int i = lo; i < hi; ++i) n_eq += ((float_key(sc[i]) & mask) == prefix);
  const int eq_before = block_exclusive_scan<kOmniTopkThreads>(n_eq, s_scan, &tot);
  int n_sel = 0, e = eq_before;
  for (int i = lo; i < hi; ++i) {
    const uint32_t km = float_key(sc[i]) & mask;
    if (km > prefix) {
      ++n_sel;
    } else if (km == prefix) {
      n_sel += (e < k_rest);
      ++e;
    }
  }
  const int at = block_exclusive_scan<kOmniTopkThreads>(n_sel, s_scan, &tot);
  int o = at;
  e = eq_before;
  for (int i = lo; i < hi; ++i) {
    const uint32_t km = float_key(sc[i]) & mask;
    bool take = km > prefix;
    if (km == prefix) take = (e++ < k_rest);
    if (take) out[o++] = i;
  }
}

// ------------------------------------------------------------------ slot attention

struct GatherParams {
  uint16_t* kv;
  int32_t* pos_pool;
  const int32_t* block_table;
  int32_t* lengths;
  int64_t num_pages;
  int32_t max_pages;
  int32_t num_kv_heads;
  const uint16_t* q;      // [num_req][Hq][D]
  const uint16_t* k_new;  // [num_req][Hkv][D] or null
  const uint16_t* v_new;
  const int32_t* new_pos;
  const int32_t* sel;     // [num_req][count]
  int32_t count;
  int32_t max_len;
  float scale_log2;       // scale * log2(e)
  float* out;             // [num_req][Hq][D]
  float* lse;             // [num_req][Hq] or null
  int32_t* dev_err;
};

// Cross-lane steps of the gather pass, all in VALU (DPP and permlane swaps,
// no LDS permutes).  row8_sum: the sum over each group of 8 lanes, in all 8
// (quad sums, then each lane adds the mirror lane of its half-row, which
// holds the other quad's sum: the pairs of an xor-1/2/4 butterfly, so the
// same rounding).  lane8_max: the maximum over the 8 lanes of equal lane % 8
// (bit 3 by a rotation of each 16-lane row by 8, bits 5 and 4 by permlane
// swaps).
constexpr int kRowHalfMirror = 0x141;  // DPP row_half_mirror: lane i of 8 reads lane 7 - i
constexpr int kRowRor8 = 0x128;        // DPP row_ror:8: lane i of 16 reads lane (i + 8) % 16
__device__ __forceinline__ float row8_sum(float v) {
  v = quad_sum(v);
  return v + dpp_f<kRowHalfMirror>(v);
}
__device__ __forceinline__ float lane8_sum(float v) {
  v += dpp_f<kRowRor8>(v);
  const uint32_t b = __float_as_uint(v);
  const auto h = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  const float y = __uint_as_float(h[0]) + __uint_as_float(h[1]);
  const uint32_t c = __float_as_uint(y);
  const auto r = __builtin_amdgcn_permlane16_swap(c, c, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float lane8_max(float v) {
  v = fmaxf(v, dpp_f<kRowRor8>(v));
  const uint32_t b = __float_as_uint(v);
  const auto h = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  const float y = fmaxf(__uint_as_float(h[0]), __uint_as_float(h[1]));
  const uint32_t c = __float_as_uint(y);
  const auto r = __builtin_amdgcn_permlane16_swap(c, c, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

typedef uint32_t gather_u32x4 __attribute__((ext_vector_type(4)));

template <int D>
struct GatherRow {
  static constexpr int QW = D / 16;  // 32-bit words of a key row per lane (8 lanes per row)
  static constexpr int VW = D / 64;  // value columns per lane
};

template <int D, int G, int NT>
__global__ __launch_bounds__(NT, (G >= 4 ? 2 : 4) * kGatherThreads / NT) void gather_attend_kernel(const GatherParams p) {
  constexpr int kGatherWaves = NT / kWave;
  constexpr int QW = GatherRow<D>::QW;
  constexpr int VC = GatherRow<D>::VW;
  __shared__ uint32_t s_row[kGatherMaxSel];
  __shared__ float s_w[kGatherWaves][8][G];
  __shared__ float s_m[kGatherWaves][G], s_l[kGatherWaves][G];
  __shared__ float s_o[kGatherWaves][G][D];
  __shared__ int s_scan[kGatherWaves + 1];
  __shared__ int s_red[kGatherWaves];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wv = tid / kWave;
  const int unit = blockIdx.x;
  const int req = unit / p.num_kv_heads;
  const int kvh = unit % p.num_kv_heads;
  const int Hq = p.num_kv_heads * G;
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int L0 = p.lengths[unit];
  const bool append = p.k_new != nullptr;
  float* o_out = p.out + ((size_t)req * Hq + (size_t)kvh * G) * D;

  // ---- append: the new token's row, position and the length
  int fail = 0;
  if (L0 < 0 || L0 + (append ? 1 : 0) > p.max_len) fail = SE_DEVERR_BAD_LENGTH;
  else if (append && L0 >= p.max_pages * kPage) fail = SE_DEVERR_CAPACITY;
  const int L = L0 + (append ? 1 : 0);
  if (!fail && append) {
    const int ph = bt[L0 >> 4];
    if (ph < 0 || (int64_t)ph >= p.num_pages) {
      fail = SE_DEVERR_BAD_PAGE;
    } else if (wv == 0) {
      const size_t krow = ((size_t)ph * 2 * kPage + (L0 & (kPage - 1))) * D;
      const uint16_t* ks = p.k_new + ((size_t)req * p.num_kv_heads + kvh) * D;
      const uint16_t* vs = p.v_new + ((size_t)req * p.num_kv_heads + kvh) * D;
      for (int c = lane; c < D; c += kWave) {
        p.kv[krow + c] = ks[c];
        p.kv[krow + (size_t)kPage * D + c] = vs[c];
      }
      if (lane == 0) p.pos_pool[(size_t)ph * kPage + (L0 & (kPage - 1))] = p.new_pos[req];
    }
  }
  if (fail) {
    if (tid == 0) set_error(p.dev_err, fail);
    for (int i = tid; i < G * D; i += NT) o_out[i] = 0.f;
    if (p.lse != nullptr && tid < G) p.lse[(size_t)req * Hq + kvh * G + tid] = -INFINITY;
    return;
  }

  // ---- queries (loaded first, so that their latency overlaps the row
  // translation): lane (row r8 = lane/8, c8 = lane%8) holds columns [c8*D/8, ...)
  // of the G rows
  const int c8 = lane & 7;
  const int r8 = lane >> 3;
  uint32_t qr[G][QW];
  {
    const uint16_t* qb = p.q + ((size_t)req * Hq + (size_t)kvh * G) * D + c8 * (D / 8);
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < QW; i += 4) {
        const uint4 t = *reinterpret_cast<const uint4*>(qb + (size_t)g * D + 2 * i);
        qr[g][i] = t.x;
        qr[g][i + 1] = t.y;
        qr[g][i + 2] = t.z;
        qr[g][i + 3] = t.w;
      }
  }
  // ---- the selected rows (entries < 0 skipped; at or past L reported and
  // skipped), 2 * NT entries a round: a thread's two entries (c0 + tid and
  // c0 + NT + tid) and their page-table entries are loaded together, and one
  // block scan of both counts (16 bits each in one int; a count is at most NT)
  // places the rows in selection order
  int n_sel = 0, bad_sel = 0, bad_page = 0;
  const int32_t* sel = p.sel + (size_t)req * p.count;
  for (int c0 = 0; c0 < p.count; c0 += 2 * NT) {
    int s2[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int i = c0 + k * NT + tid;
      s2[k] = i < p.count ? sel[i] : -1;
    }
    int ph2[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) ph2[k] = (s2[k] >= 0 && s2[k] < L) ? bt[s2[k] >> 4] : 0;
    uint32_t row2[2];
    bool ok2[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int s_ = s2[k];
      bool ok = s_ >= 0 && s_ < L;
      bad_sel |= (s_ >= L);
      row2[k] = 0;
      if (ok) {
        if (append && s_ == L0) {
          row2[k] = kNewRow;
        } else if (ph2[k] < 0 || (int64_t)ph2[k] >= p.num_pages) {
          ok = false;
          bad_page = 1;
        } else {
          row2[k] = (uint32_t)ph2[k] * 2 * kPage + (uint32_t)(s_ & (kPage - 1));
        }
      }
      ok2[k] = ok;
    }
    int tot;
    const int at = block_exclusive_scan<NT>((ok2[0] ? 1 : 0) | (ok2[1] ? 1 << 16 : 0), s_scan, &tot);
    const int tot0 = tot & 0xFFFF;
    const int at0 = n_sel + (at & 0xFFFF), at1 = n_sel + tot0 + (at >> 16);
    if (ok2[0] && at0 < kGatherMaxSel) s_row[at0] = row2[0];
    if (ok2[1] && at1 < kGatherMaxSel) s_row[at1] = row2[1];
    n_sel += tot0 + (tot >> 16);
  }
  if (tid == 0 && bad_sel) set_error(p.dev_err, SE_DEVERR_BAD_SELECTION);
  {
    const int bp = block_reduce<NT>(bad_page, s_red, [](int a, int c) { return a | c; });
    if (bp && tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
  }
  n_sel = min(n_sel, kGatherMaxSel);
  __syncthreads();  // the row list and the appended row are complete
  if (append && tid == 0) p.lengths[unit] = L;

  const uint16_t* knew = append ? p.k_new + ((size_t)req * p.num_kv_heads + kvh) * D : nullptr;
  const uint16_t* vnew = append ? p.v_new + ((size_t)req * p.num_kv_heads + kvh) * D : nullptr;

  // the wavefront's share of the rows, in passes of 8
  const int per = ceil_div_dev(n_sel, kGatherWaves);
  const int rb = min(n_sel, wv * per), re = min(n_sel, rb + per);
  const int n_pass = ceil_div_dev(re - rb, 8);

  struct Buf {
    uint32_t k[QW];
    uint32_t v[8];
  };
  auto load = [&](int ps, Buf& bf) {
    const int e = min(rb + ps * 8 + r8, re - 1);
    const uint32_t row = s_row[max(e, 0)];
    const uint16_t* ksrc = row == kNewRow ? knew : p.kv + (size_t)row * D;
    // rows are read once: nontemporal loads (as the decode stream's)
    const gather_u32x4* k4 = reinterpret_cast<const gather_u32x4*>(ksrc + c8 * (D / 8));
#pragma unroll
    for (int i = 0; i < QW; i += 4) {
      const gather_u32x4 t = __builtin_nontemporal_load(k4 + i / 4);
      bf.k[i] = t.x;
      bf.k[i + 1] = t.y;
      bf.k[i + 2] = t.z;
      bf.k[i + 3] = t.w;
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int er = min(rb + ps * 8 + r, re - 1);
      const uint32_t vr = __builtin_amdgcn_readfirstlane(s_row[max(er, 0)]);  // one row per wavefront
      const uint16_t* vsrc = vr == kNewRow ? vnew : p.kv + ((size_t)vr + kPage) * D;
      if (VC == 2)
        bf.v[r] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(vsrc) + lane);
      else
        bf.v[r] = __builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(vsrc) + lane);
    }
  };

  float m[G], l[G], acc[G][VC];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int c = 0; c < VC; ++c) acc[g][c] = 0.f;
  }
  // one pass: logits of row r8 for every head (reduced over the row's 8
  // lanes), the pass maximum per head, rescale, weights through LDS, values
  auto pass = [&](int ps, const Buf& cur) {
    float z[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < QW; ++i) a = dot2bf16(qr[g][i], cur.k[i], a);
      a = row8_sum(a);
      z[g] = rb + ps * 8 + r8 < re ? a * p.scale_log2 : -INFINITY;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = z[g];
      mx = lane8_max(mx);
      const float mn = fmaxf(m[g], mx);
      const float corr = fast_exp2(m[g] - mn);  // m = -inf at first: 0
      m[g] = mn;
      const float w = fast_exp2(z[g] - mn);
      if (c8 == 0) s_w[wv][r8][g] = w;
      l[g] = fmaf(l[g], corr, w);  // row r8's share (the row's 8 lanes hold the same)
#pragma unroll
      for (int c = 0; c < VC; ++c) acc[g][c] *= corr;
    }
    wave_lds_sync();
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      float vf[VC];
      if (VC == 2) {
        vf[0] = bf16lo(cur.v[r]);
        if (VC > 1) vf[VC - 1] = bf16hi(cur.v[r]);
      } else {
        vf[0] = bf16f((uint16_t)cur.v[r]);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float wgt = s_w[wv][r][g];
#pragma unroll
        for (int c = 0; c < VC; ++c) acc[g][c] = fmaf(wgt, vf[c], acc[g][c]);
      }
    }
    wave_lds_sync();
  };
  // three buffers, two passes in flight while one is reduced; loads past the
  // share re-read its last row, so every step issues the same loads and the
  // waits stay partial (the loop is unrolled by three: every buffer keeps its
  // registers)
  if (n_pass > 0) {
    Buf b0, b1, b2;
    load(0, b0);
    load(1, b1);
    load(2, b2);
    for (int ps = 0; ps < n_pass; ps += 3) {
      pass(ps, b0);
      load(ps + 3, b0);
      if (ps + 1 < n_pass) pass(ps + 1, b1);
      load(ps + 4, b1);
      if (ps + 2 < n_pass) pass(ps + 2, b2);
      load(ps + 5, b2);
    }
  }
  // ---- combine the wavefronts (l: the sum of the 8 row lanes' shares)
#pragma unroll
  for (int g = 0; g < G; ++g) {
    l[g] = lane8_sum(l[g]);
    if (lane == 0) {
      s_m[wv][g] = m[g];
      s_l[wv][g] = l[g];
    }
#pragma unroll
    for (int c = 0; c < VC; ++c) s_o[wv][g][lane * VC + c] = acc[g][c];
  }
  __syncthreads();
  for (int i = tid; i < G * D; i += NT) {
    const int g = i / D, col = i % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kGatherWaves; ++w) M = fmaxf(M, s_m[w][g]);
    float lsum = 0.f, o = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kGatherWaves; ++w) {
        const float f = s_m[w][g] == -INFINITY ? 0.f : fast_exp2(s_m[w][g] - M);
        lsum += s_l[w][g] * f;
        o += s_o[w][g][col] * f;
      }
    }
    o_out[(size_t)g * D + col] = lsum > 0.f ? o / lsum : 0.f;
    if (col == 0 && p.lse != nullptr)
      p.lse[(size_t)req * Hq + kvh * G + g] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
  }
}

// 1024 threads when the units take at most one work-group per compute unit
// (groups of up to 4 query heads: a group of 8 would not fit 128 registers)
template <int D>
void launch_gather_d(const GatherParams& p, int units, int G, hipStream_t s) {
  constexpr int NW = kGatherThreadsWide, N = kGatherThreads;
  const bool wide = units <= 256;
  switch (G) {
    case 1:
      if (wide) hipLaunchKernelGGL((gather_attend_kernel<D, 1, NW>), dim3(units), dim3(NW), 0, s, p);
      else hipLaunchKernelGGL((gather_attend_kernel<D, 1, N>), dim3(units), dim3(N), 0, s, p);
      break;
    case 2:
      if (wide) hipLaunchKernelGGL((gather_attend_kernel<D, 2, NW>), dim3(units), dim3(NW), 0, s, p);
      else hipLaunchKernelGGL((gather_attend_kernel<D, 2, N>), dim3(units), dim3(N), 0, s, p);
      break;
    case 4:
      if (wide) hipLaunchKernelGGL((gather_attend_kernel<D, 4, NW>), dim3(units), dim3(NW), 0, s, p);
      else hipLaunchKernelGGL((gather_attend_kernel<D, 4, N>), dim3(units), dim3(N), 0, s, p);
      break;
    default: hipLaunchKernelGGL((gather_attend_kernel<D, 8, N>), dim3(units), dim3(N), 0, s, p); break;
  }
}

}  // namespace se

using namespace se;

size_t se_omnikv_workspace_bytes(int32_t num_req, int32_t max_len) {
  if (num_req <= 0 || max_len <= 0) return 0;
  return (size_t)num_req * align_up((size_t)max_len, 64) * sizeof(float);
}

extern "C" se_status se_omnikv_select(const se_kv_view* kv, int32_t q_per_kv, const float* logits,
                                      int32_t logits_stride, int32_t budget, int32_t max_len,
                                      int32_t* sel_slots, void* ws, size_t ws_bytes, int32_t* dev_err,
                                      hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (logits == nullptr || sel_slots == nullptr || dev_err == nullptr) return SE_ERR_INVALID_ARGUMENT;
  if (q_per_kv < 1 || q_per_kv > 8 || budget < 1 || max_len < 1 || logits_stride < max_len)
    return SE_ERR_INVALID_ARGUMENT;
  if (budget > kGatherMaxSel) return SE_ERR_UNSUPPORTED;
  const int num_req = kv->num_units / kv->num_kv_heads;
  if (ws == nullptr || ws_bytes < se_omnikv_workspace_bytes(num_req, max_len)) return SE_ERR_WORKSPACE;
  OmniSelectParams p;
  p.logits = logits;
  p.stride = logits_stride;
  p.lengths = kv->lengths;
  p.num_req = num_req;
  p.num_kv_heads = kv->num_kv_heads;
  p.q_per_kv = q_per_kv;
  p.budget = budget;
  p.max_len = max_len;
  p.ws_stride = (int32_t)align_up((size_t)max_len, 64);
  p.vec4 = (reinterpret_cast<uintptr_t>(logits) % 16 == 0 && logits_stride % 4 == 0 &&
            reinterpret_cast<uintptr_t>(ws) % 16 == 0) ? 1 : 0;
  p.scores = static_cast<float*>(ws);
  p.sel = sel_slots;
  p.dev_err = dev_err;
  const int chunks = (int)ceil_div(max_len, kOmniScoreThreads * kOmniScoreSlots);
  hipLaunchKernelGGL(omnikv_score_kernel, dim3(chunks, num_req), dim3(kOmniScoreThreads), 0, stream, p);
  hipLaunchKernelGGL(omnikv_topk_kernel, dim3(num_req), dim3(kOmniTopkThreads), 0, stream, p);
  return launch_status();
}

extern "C" se_status se_attend_slots(const se_kv_view* kv, int32_t q_per_kv, const void* q, const void* k_new,
                                     const void* v_new, const int32_t* new_pos, const int32_t* sel_slots,
                                     int32_t sel_count, float scale, int32_t max_len, float* out, float* lse,
                                     int32_t* dev_err, hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->kv_pool == nullptr || kv->pos_pool == nullptr || q == nullptr || sel_slots == nullptr ||
      out == nullptr || dev_err == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if ((k_new == nullptr) != (v_new == nullptr) || (k_new != nullptr && new_pos == nullptr))
    return SE_ERR_INVALID_ARGUMENT;
  if (sel_count < 1 || max_len < 1 || !(scale > 0.f)) return SE_ERR_INVALID_ARGUMENT;
  if (q_per_kv != 1 && q_per_kv != 2 && q_per_kv != 4 && q_per_kv != 8) return SE_ERR_UNSUPPORTED;
  if (sel_count > kGatherMaxSel) return SE_ERR_UNSUPPORTED;
  if (kv->num_pages > ((int64_t)1 << 27)) return SE_ERR_UNSUPPORTED;  // row indices are 32-bit
  GatherParams p;
  p.kv = static_cast<uint16_t*>(kv->kv_pool);
  p.pos_pool = kv->pos_pool;
  p.block_table = kv->block_table;
  p.lengths = kv->lengths;
  p.num_pages = kv->num_pages;
  p.max_pages = kv->max_pages;
  p.num_kv_heads = kv->num_kv_heads;
  p.q = static_cast<const uint16_t*>(q);
  p.k_new = static_cast<const uint16_t*>(k_new);
  p.v_new = static_cast<const uint16_t*>(v_new);
  p.new_pos = new_pos;
  p.sel = sel_slots;
  p.count = sel_count;
  p.max_len = max_len;
  p.scale_log2 = scale * kLog2e;
  p.out = out;
  p.lse = lse;
  p.dev_err = dev_err;
  if (kv->head_dim == 128)
    launch_gather_d<128>(p, kv->num_units, q_per_kv, stream);
  else
    launch_gather_d<64>(p, kv->num_units, q_per_kv, stream);
  return launch_status();
}
