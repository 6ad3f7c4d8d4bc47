// se_snapkv_compact: SnapKV prompt compaction (Appendix A.3, "SnapKV: Prompt
// Selection from an Observation Window", eqs. background-snapkv-score and
// background-snapkv-retention), applied to a unit's prompt after its last
// prefill chunk (Section 3.1, finish_step during prefill).
//
// Scoring runs one work-group of eight wavefronts per unit, two work-groups
// per compute unit.  The w observation queries of the unit's G heads form
// R = w*G rows; up to 128 of them sit in four row groups of 32 (more rows:
// see the accumulate mode below); wavefront v holds row group v % 4 in
// registers as MFMA A operands (bf16 16x16x32 tiles: lane l holds
// row l%16 and contraction indices 8*(l/16)..+7 of each 32-wide step) and
// takes the pages of key half v / 4 of every stage.  The unit's key pages
// stream through a two-stage LDS ring of four pages a stage: the work-group
// loads every page as coalesced 16-byte pieces, two stages ahead, into
// registers, and writes them to LDS with the piece index XORed with the key
// so that the B-operand reads (lane l: key l%16) hit distinct banks.  A page
// (16 keys) is one B tile; the 16x16 output tile gives lane l the logits of
// key l%16 against rows 4*(l/16)..+3 of each row tile.
//   pass 1  row normalisers: every lane keeps, per row, a reference and the
//           sum of exp2(c*z - reference) over its keys (c = scale*log2 e); a
//           reference moves only when a logit passes it by more than kLazy,
//           so most pages cost one fma, one max, one exp2 and one add per
//           logit.  Merging the 16 key lanes and the two key halves of a row
//           gives bias = log2 of the row's softmax denominator.
//   pass 2  u(j) = sum over rows of exp2(c*z - bias) for the candidate keys:
//           in-lane over the lane's rows, across the lane groups with permlane
//           swaps; each wavefront leaves its row group's sums in LDS, and once
//           the stage has passed a wavefront adds the four row groups of each
//           key of one page and writes u to the workspace.
//   pool    s(j) = max of u over the candidates within kappa/2 positions of j,
//           through LDS chunks with a halo; s goes to the score field of the
//           candidates and 0 to the window's, and a slot order that is not
//           strictly increasing in position is reported.
// The keys are read twice: the weights need the row's normaliser, which
// depends on every key, and keeping the logits (R floats per key) would cost
// more than re-reading the key (2*d bytes).  The causal mask touches only the
// last pages (window keys); slots past the length are masked there too.
// Retention and compaction are then H2O's kernel (launch_evict) with the
// window as its recent set.
//
// SnapKV with more than 128 rows (up to 1024) runs the kernel in the
// accumulate mode of the chunk scoring below: each row block of 128 rows
// writes its partial u per key (the causal mask reaches only window keys),
// and snapkv_pool_kernel adds the blocks in block order and pools over the
// candidates.
//
// H2O chunk scoring (se_h2o_prefill_chunk) with 257 .. 512 scoring rows runs
// the key-split kernels further below; with other row counts it runs the same
// kernel over every key with the causal mask in both passes, one row block of
// up to 128 scoring rows
// per work-group (grid.y), one work-group per CU; a block of 128 rows sits in
// two row groups of 64 (four row tiles per wavefront, each stage's four pages
// split over the four wavefronts of a row group), so each key piece read from
// LDS feeds four MFMA row tiles instead of two.  There the stages made only
// of pages below the window run pipelined: stage j's MFMAs are issued in the
// same branch-free block as the exponentials of stage j - 1's logits (the two
// stages' logits alternate between two register sets), and four stages of
// loads are in flight; the remaining pages go through the per-page path.
#include <algorithm>

#include "evict_core.h"

namespace se {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kSnapThreads = 512;
constexpr int kSnapWaves = kSnapThreads / kWave;
constexpr int kSnapRowGroups = 4;       // of up to 32 rows (SnapKV); H2O chunk scoring: 2 of 64
constexpr int kSnapMaxRows = 128;
constexpr int kPrefillBlockRows = 128;  // rows of a work-group in H2O chunk scoring
constexpr int kSnapMaxHalf = 15;        // kappa <= 31
constexpr int kSnapMaxPages = 8192;     // pages per unit (131072 slots)
constexpr int kSnapStagePages = 4;      // pages per ring stage
constexpr int kSnapBatches = 2;         // stages in flight per thread
constexpr int kSnapPoolChunk = 2048;    // slots pooled per LDS round
constexpr int kSnapHalo = kSnapMaxHalf + 1;
constexpr float kLazy = 20.f;           // log2 headroom before a reference moves
constexpr float kRefInit = -1e30f;      // finite: differences stay defined

struct SnapParams {
  const uint16_t* kv;
  const int32_t* pos_pool;
  float* score_pool;
  const int32_t* block_table;
  const int32_t* lengths;
  const uint16_t* q;  // bf16 [num_req][w][Hq][d]
  float* u;           // fp32 [num_units][u_stride]
  int64_t num_pages;
  int32_t max_pages;
  int32_t num_kv_heads;
  int32_t q_per_kv;
  int32_t w;
  int32_t half;
  int32_t budget;
  int32_t max_len;
  int32_t u_stride;
  int32_t n_rb;       // row blocks of kSnapMaxRows rows (grid.y)
  int32_t chunk;      // H2O prefill: the chunk's slots (the last ones); 0 for SnapKV
  int32_t vec4;       // H2O prefill: score pool and workspace 16-byte aligned
  int32_t snap_wide;  // SnapKV scored in row blocks (accumulate mode): skip units at or under the budget
  float c;  // scale * log2(e)
  int32_t* dev_err;
};

__device__ __forceinline__ f32x4_t mfma16x16x32(const uint4& a, const uint4& b, f32x4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                 acc, 0, 0, 0);
}

// The K block of a page in LDS: 16 keys of D/8 16-byte pieces; piece c of key
// k sits at column c ^ (k mod D/8).
template <int D>
__device__ __forceinline__ int ring_offset(int key, int piece) {
  constexpr int PC = D / 8;
  return key * (2 * D) + ((piece ^ (key & (PC - 1))) << 4);
}

// Streams pages [pb, pe) of the unit through the LDS ring; body(j, slot)
// runs once per stage of kSnapStagePages pages (stage j holds pages
// pb + j*kSnapStagePages ..., in ring slot j % 2), every thread of the
// work-group taking part.  Each thread keeps kSnapBatches stages of its
// pieces in flight in registers (a stage's loads are issued kSnapBatches - 1
// stages before it is written to LDS); loads past the range re-read its last
// page.  The loop is unrolled by kSnapBatches so that every batch keeps its
// registers, and has no exit between its steps, so the loop head is reached
// with the same loads in flight on every path.
// A block-table entry at a wavefront-uniform index, as a scalar load: the
// table is read-only for the whole launch, so it may go through the constant
// address space.
typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;
__device__ __forceinline__ int bt_entry(const int32_t* bt, int i) {
  return ((const_i32_ptr)bt)[__builtin_amdgcn_readfirstlane(i)];
}

template <int D, int NB, int NT = kSnapThreads, typename Body>
__device__ __forceinline__ void stream_stages(const SnapParams& p, const int32_t* bt, uint8_t* ring, int pb, int pe,
                                              Body body) {
  constexpr int S = kSnapStagePages;
  constexpr int PB = 32 * D;                       // K bytes of a page
  constexpr int PC = D / 8;                        // 16-byte pieces per key
  constexpr int PT = S * 2 * D / NT;               // pieces per thread per stage
  static_assert(NB % 2 == 0, "ring slots alternate within the unrolled loop");
  static_assert(PT >= 1 && PT * NT == S * 2 * D, "whole pages per stage");
  const int n_st = ceil_div_dev(pe - pb, S);
  if (n_st <= 0) return;
  // piece g = threadIdx.x + q * NT of a stage: page g / (2D), piece g % (2D)
  int pg_of[PT], off_of[PT], lds_of[PT];
#pragma unroll
  for (int q = 0; q < PT; ++q) {
    const int g = (int)threadIdx.x + q * NT;
    const int pp = g / (2 * D);
    const int t = g % (2 * D);
    pg_of[q] = __builtin_amdgcn_readfirstlane(pp);  // 2D is a multiple of the wavefront
    off_of[q] = t * 8;
    lds_of[q] = pp * PB + ring_offset<D>(t / PC, t % PC);
  }
  auto load = [&](u32x4_t(&r)[PT], int st) {
#pragma unroll
    for (int q = 0; q < PT; ++q) {
      const int pg = min(pb + st * S + pg_of[q], pe - 1);  // the same in every lane of a wavefront
      r[q] = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4_t*>(p.kv + (size_t)bt_entry(bt, pg) * 2 * kPage * D + off_of[q]));
    }
  };
  auto store = [&](const u32x4_t(&r)[PT], int slot) {
#pragma unroll
    for (int q = 0; q < PT; ++q) *reinterpret_cast<u32x4_t*>(ring + slot * S * PB + lds_of[q]) = r[q];
  };
  u32x4_t r[NB][PT];
  load(r[0], 0);
  store(r[0], 0);
#pragma unroll
  for (int b = 1; b < NB; ++b) {
    asm volatile("" ::: "memory");  // issue order: stage b before stage b + 1
    load(r[b], b);
  }
  asm volatile("" ::: "memory");
  load(r[0], NB);
  __syncthreads();
  for (int j = 0; j < n_st; j += NB) {
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      store(r[(k + 1) % NB], (k + 1) & 1);  // stage j + k + 1
      load(r[(k + 1) % NB], j + k + 1 + NB);
      if (j + k < n_st) body(j + k, k & 1);
      __syncthreads();
    }
  }
}

// Logits of the page at `page` (LDS) against the wavefront's row tiles:
// acc[T][r] is row tile T, row 4*(lane/16) + r, against key lane%16.
template <int D, int RTW>
__device__ __forceinline__ void page_logits(const uint4 (&qa)[RTW][D / 32], const uint8_t* page, f32x4_t (&acc)[RTW]) {
  constexpr int KS = D / 32;
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane >> 4;
  const int col = lane & 15;
  uint4 kb[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) kb[s] = *reinterpret_cast<const uint4*>(page + ring_offset<D>(col, 4 * s + grp));
#pragma unroll
  for (int T = 0; T < RTW; ++T) acc[T] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int T = 0; T < RTW; ++T) acc[T] = mfma16x16x32(qa[T][s], kb[s], acc[T]);
}

// Sum over the four 16-lane groups of a wavefront, in every lane (lane l gets
// the sum of lanes l%16, l%16 + 16, l%16 + 32, l%16 + 48): the upper and lower
// halves, then the odd and even 16-lane rows, exchanged by permlane swaps.
__device__ __forceinline__ float lane_group_sum(float x) {
  const uint32_t b = __float_as_uint(x);
  const auto h = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  const float y = __uint_as_float(h[0]) + __uint_as_float(h[1]);
  const uint32_t c = __float_as_uint(y);
  const auto r = __builtin_amdgcn_permlane16_swap(c, c, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// (ref, sum) pairs merged: the sum re-expressed against the larger reference.
__device__ __forceinline__ void merge_norm(float& ref, float& sum, float ref2, float sum2) {
  const float m = fmaxf(ref, ref2);
  sum = sum * fast_exp2(ref - m) + sum2 * fast_exp2(ref2 - m);
  ref = m;
}

// Max pooling (SnapKV's s): s(j) = max of u over the candidates (slots [0,
// n_lim)) within `half` positions of j, 0 on the window, written to the score
// field, through LDS chunks with a halo; a slot order that is not strictly
// increasing in position is reported.  u_of(j) gives u(j) for j < n_lim.
template <typename UFn>
__device__ __forceinline__ void snapkv_pool(const SnapParams& p, const int32_t* bt, int L, int n_lim, UFn u_of,
                                            uint8_t* scratch, int* s_red) {
  const int tid = threadIdx.x;
  const int half = p.half;
  int32_t* s_pos = reinterpret_cast<int32_t*>(scratch);
  float* s_u = reinterpret_cast<float*>(scratch) + kSnapPoolChunk + 2 * kSnapHalo;
  int bad_pos = 0;
  for (int c0 = 0; c0 < L; c0 += kSnapPoolChunk) {
    for (int i = tid; i < kSnapPoolChunk + 2 * kSnapHalo; i += kSnapThreads) {
      const int j = c0 - kSnapHalo + i;
      int32_t pj = 0;
      float uj = -INFINITY;
      if (j >= 0 && j < L) {
        pj = p.pos_pool[(size_t)bt[j >> 4] * kPage + (j & (kPage - 1))];
        if (j < n_lim) uj = u_of(j);
      }
      s_pos[i] = pj;
      s_u[i] = uj;
    }
    __syncthreads();
    for (int i = tid; i < kSnapPoolChunk && c0 + i < L; i += kSnapThreads) {
      const int j = c0 + i;
      const int x = i + kSnapHalo;
      const int32_t pj = s_pos[x];
      if (j > 0 && s_pos[x - 1] >= pj) bad_pos = 1;
      float s = 0.f;
      if (j < n_lim) {
        s = s_u[x];
        for (int k = 1; k <= half; ++k) {
          // slots outside [0, n_lim) hold -inf; positions strictly increase, so
          // the candidates within half positions are within half slots
          if ((int64_t)pj - s_pos[x - k] <= half) s = fmaxf(s, s_u[x - k]);
          if ((int64_t)s_pos[x + k] - pj <= half) s = fmaxf(s, s_u[x + k]);
        }
      }
      p.score_pool[(size_t)bt[j >> 4] * kPage + (j & (kPage - 1))] = s;
    }
    __syncthreads();
  }
  bad_pos = block_reduce<kSnapThreads>(bad_pos, s_red, [](int a, int b) { return a | b; });
  if (bad_pos && tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_POSITIONS);
}


// RTW: 16-row tiles per row group (rows of group g: [16*RTW*g, 16*RTW*(g+1)) of
// the work-group's row block blockIdx.y).  kAccum: H2O chunk scoring -- u over
// every key (the window keys with their causal mask) into the row block's
// partial row of the workspace, no pooling; otherwise SnapKV.
template <int D, int RTW, bool kAccum, bool kPipe, int kOcc, int NRG>
__global__ __launch_bounds__(kSnapThreads, kOcc) void snapkv_score_kernel(const SnapParams p) {
  // NRG row groups of 16 * RTW rows; the wavefronts of one row group split
  // each stage's pages (NKH key parts of H pages)
  constexpr int NKH = kSnapWaves / NRG;
  static_assert(NKH * NRG == kSnapWaves && kSnapStagePages % NKH == 0, "wavefront layout");
  // stages in flight per thread: four when one work-group holds the CU
  constexpr int kNB = kOcc <= 2 ? 2 * kSnapBatches : kSnapBatches;
  constexpr int KS = D / 32;
  constexpr int S = kSnapStagePages;
  constexpr int H = kSnapStagePages / NKH;
  constexpr int PB = 32 * D;
  constexpr int kRingBytes = 2 * S * 32 * 128;  // sized for head_dim 128
  static_assert(kRingBytes >= (kSnapPoolChunk + 2 * kSnapHalo) * 8, "the pool chunk reuses the ring");
  __shared__ __attribute__((aligned(16))) uint8_t s_ring[kRingBytes];
  __shared__ float s_up[2][S][NRG][kPage];     // [stage parity][page][row group][key]
  __shared__ float s_norm[NKH][2][kSnapMaxRows];   // [key part][ref, sum][row]
  __shared__ int s_red[kSnapWaves];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int grp = lane >> 4;
  const int col = lane & 15;
  const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int rg = wv % NRG;
  const int kh = wv / NRG;
  const int unit = blockIdx.x;
  const int L = p.lengths[unit];
  if ((!kAccum || p.snap_wide) && L <= p.budget) return;  // the prompt already fits: nothing to score or evict
  if (L > p.max_len || L > p.max_pages * kPage || L > kSnapMaxPages * kPage || (kAccum && L < p.chunk)) {
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return;
  }
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int n_pages = ceil_div_dev(L, kPage);
  {
    int bad = 0;
    for (int i = tid; i < n_pages; i += kSnapThreads) {
      const int ph = bt[i];
      bad |= (ph < 0 || (int64_t)ph >= p.num_pages);
    }
    bad = block_reduce<kSnapThreads>(bad, s_red, [](int a, int b) { return a | b; });
    if (bad) {
      if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
      return;
    }
  }
  const int w = p.w;
  const int G = p.q_per_kv;
  const int R = w * G;
  // SnapKV: u over the candidates (L > budget >= w, so at least one); H2O: every key
  const int n_lim = kAccum ? L : L - w;
  const int row0 = 16 * RTW * rg;                // within the row block
  const int rbase = (kAccum ? kPrefillBlockRows : kSnapMaxRows) * blockIdx.y;  // the row block's first row

  // ---- the row group's observation queries (A operands); rows past R are zero
  uint4 qa[RTW][KS];
  {
    const int req = unit / p.num_kv_heads;
    const int kvh = unit % p.num_kv_heads;
    const int hq = p.num_kv_heads * G;
#pragma unroll
    for (int T = 0; T < RTW; ++T) {
      const int row = rbase + row0 + 16 * T + col;
      const int t = row / G;
      const int g = row - t * G;
      const uint16_t* src = p.q + (((size_t)req * w + t) * hq + (size_t)kvh * G + g) * D + 8 * grp;
#pragma unroll
      for (int s = 0; s < KS; ++s)
        qa[T][s] = row < R ? *reinterpret_cast<const uint4*>(src + 32 * s) : uint4{0u, 0u, 0u, 0u};
    }
  }
  // the queries arrive before the page stream starts, so that the stream's
  // waits count page loads only
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int s = 0; s < KS; ++s)
      asm volatile("" : "+v"(qa[T][s].x), "+v"(qa[T][s].y), "+v"(qa[T][s].z), "+v"(qa[T][s].w));
  const float c = p.c;
  // pages [0, p_full) hold only keys every row sees (slot <= L - w)
  const int p_full = (L - w + 1) / kPage;

  // ---- pass 1: row normalisers
  float ref[RTW][4], sum[RTW][4];
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ref[T][r] = kRefInit;
      sum[T][r] = 0.f;
    }
  // one page's logits into the references and sums
  auto norm_page = [&](const f32x4_t(&a)[RTW]) {
    float dmax = -INFINITY;
    float d[RTW][4];
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        d[T][r] = fmaf(a[T][r], c, -ref[T][r]);
        dmax = fmaxf(dmax, d[T][r]);
      }
    if (__builtin_amdgcn_ballot_w64(dmax > kLazy) != 0) {
      // rare: raise the references of the wavefront's rows to their logits
#pragma unroll
      for (int T = 0; T < RTW; ++T)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float zc = a[T][r] * c;
          const float m = fmaxf(ref[T][r], zc);
          sum[T][r] *= fast_exp2(ref[T][r] - m);
          d[T][r] = zc - m;
          ref[T][r] = m;
        }
    }
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) sum[T][r] += fast_exp2(d[T][r]);
  };
  // the causal mask of a page holding window keys: key j is seen by the rows
  // of window position t iff j <= L - w + t (so j < L); padded rows see nothing
  auto causal_mask = [&](f32x4_t(&a)[RTW], int pg, float masked) {
    const int key = pg * kPage + col;
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + row0 + 16 * T + 4 * grp + r;
        const int lim = row < R ? L - w + row / G : -1;
        if (key > lim) a[T][r] = masked;
      }
  };
  // Whole stages of pages below p_full run pipelined: the stage's MFMAs are
  // issued beside the exponentials of the previous stage's logits, in one
  // branch-free block (the reference check of a stage is one ballot after
  // its exponentials; the rare raise redoes the stage page by page).
  const int pe1 = kPipe ? min(p_full, n_pages) / S * S : 0;
  if (kPipe) {
    // the logits of two stages: a stage in ring slot k leaves its logits in
    // accs[k] and reads the previous stage's from accs[k ^ 1] (the ring slot
    // is a constant in each unrolled step, so nothing is copied); -inf logits
    // add nothing
    f32x4_t accs[2][H][RTW];
#pragma unroll
    for (int i = 0; i < H; ++i)
#pragma unroll
      for (int T = 0; T < RTW; ++T) accs[1][i][T] = f32x4_t{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    auto norm_stage = [&](const f32x4_t(&prev)[H][RTW]) {
      float t[RTW][4];
      float dmax = -INFINITY;
#pragma unroll
      for (int T = 0; T < RTW; ++T)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
          for (int i = 0; i < H; ++i) {
            const float d = fmaf(prev[i][T][r], c, -ref[T][r]);
            dmax = fmaxf(dmax, d);
            t[T][r] = i == 0 ? fast_exp2(d) : t[T][r] + fast_exp2(d);
          }
        }
      // the exponentials stay here, beside the stage's MFMAs, rather than
      // sinking past the rare branch that does not use them
#pragma unroll
      for (int T = 0; T < RTW; ++T)
#pragma unroll
        for (int r = 0; r < 4; ++r) asm volatile("" ::"v"(t[T][r]));
      if (__builtin_amdgcn_ballot_w64(dmax > kLazy) != 0) {
#pragma unroll
        for (int i = 0; i < H; ++i) norm_page(prev[i]);
#pragma unroll
        for (int T = 0; T < RTW; ++T)
#pragma unroll
          for (int r = 0; r < 4; ++r) t[T][r] = 0.f;
      }
#pragma unroll
      for (int T = 0; T < RTW; ++T)
#pragma unroll
        for (int r = 0; r < 4; ++r) sum[T][r] += t[T][r];
    };
    stream_stages<D, kNB>(p, bt, s_ring, 0, pe1, [&](int j, int slot) {
#pragma unroll
      for (int i = 0; i < H; ++i) page_logits<D, RTW>(qa, s_ring + (slot * S + kh * H + i) * PB, accs[slot][i]);
      norm_stage(accs[slot ^ 1]);
    });
    if ((pe1 / S) & 1) norm_stage(accs[0]);  // the last stage
    else norm_stage(accs[1]);
  }
  // the remaining pages one at a time, masked where they hold window keys
  stream_stages<D, kNB>(p, bt, s_ring, pe1, n_pages, [&](int j, int slot) {
    // the half's logits first (independent MFMA chains), then the updates
    f32x4_t acc[H][RTW];
#pragma unroll
    for (int i = 0; i < H; ++i) page_logits<D, RTW>(qa, s_ring + (slot * S + kh * H + i) * PB, acc[i]);
#pragma unroll
    for (int i = 0; i < H; ++i) {
      const int pg = pe1 + j * S + kh * H + i;
      if (pg >= n_pages) break;
      if (pg >= p_full) causal_mask(acc[i], pg, -INFINITY);
      norm_page(acc[i]);
    }
  });
  // merge the 16 key lanes of each row, then the two key halves through LDS:
  // bias = log2 of the softmax denominator
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int m = 1; m < 16; m <<= 1)
        merge_norm(ref[T][r], sum[T][r], shfl_xor_f(ref[T][r], m), shfl_xor_f(sum[T][r], m));
      if (col == 0) {
        s_norm[kh][0][row0 + 16 * T + 4 * grp + r] = ref[T][r];
        s_norm[kh][1][row0 + 16 * T + 4 * grp + r] = sum[T][r];
      }
    }
  __syncthreads();
  float bias[RTW][4];
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = row0 + 16 * T + 4 * grp + r;  // within the block
      float m = s_norm[0][0][row], sm = s_norm[0][1][row];
#pragma unroll
      for (int h = 1; h < NKH; ++h) merge_norm(m, sm, s_norm[h][0][row], s_norm[h][1][row]);
      bias[T][r] = rbase + row < R ? m + __log2f(sm) : INFINITY;
    }

  // ---- pass 2: SnapKV: u over the candidate keys (every row sees them; no
  // mask); H2O: u over every key, the window keys masked as in pass 1
  float* u = p.u + ((size_t)unit * p.n_rb + blockIdx.y) * p.u_stride;
  const int cand_pages = ceil_div_dev(n_lim, kPage);
  // every wavefront leaves its row group's sum for each key of each page of
  // stage j in LDS; once the stage's barrier has passed, wavefront v < S adds
  // the four row groups of each key of page v (while the next stage runs, or
  // after the stream for the last stage)
  static_assert(S <= kSnapWaves, "one page of a stage per adding wavefront");
  auto flush = [&](int j) {
    if (wv < S && lane < kPage) {
      const float* up = &s_up[j & 1][wv][0][lane];
      float v = 0.f;
#pragma unroll
      for (int g = 0; g < NRG; ++g) v += up[g * kPage];
      const int key = (j * S + wv) * kPage + lane;
      if (key < n_lim) u[key] = v;
    }
  };
  // a page's weights summed over the lane's rows (a tree: independent exp2s,
  // short add chains), then over the four lane groups (rows 4*(lane/16)..+3
  // of each tile) of key lane%16
  auto page_sum = [&](const f32x4_t(&a)[RTW]) {
    float e[RTW * 4];
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) e[4 * T + r] = fast_exp2(fmaf(a[T][r], c, -bias[T][r]));
#pragma unroll
    for (int n = RTW * 4; n > 1; n >>= 1)
#pragma unroll
      for (int k = 0; k < n / 2; ++k) e[k] = e[2 * k] + e[2 * k + 1];
    return lane_group_sum(e[0]);
  };
  // Pipelined whole stages as in pass 1 (SnapKV: every candidate page; H2O:
  // the pages below p_full): stage j's MFMAs beside stage j - 1's sums, which
  // go to LDS, and stage j - 2's flush.
  const int pe2 = kPipe ? (kAccum ? min(p_full, cand_pages) : cand_pages) / S * S : 0;
  const int n1 = pe2 / S;
  if (kPipe) {
    f32x4_t accs[2][H][RTW];  // as in pass 1; -inf logits: zero weights
#pragma unroll
    for (int i = 0; i < H; ++i)
#pragma unroll
      for (int T = 0; T < RTW; ++T) accs[1][i][T] = f32x4_t{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    auto sums_to_lds = [&](int j, const f32x4_t(&prev)[H][RTW]) {  // the sums of stage j
      float us[H];
#pragma unroll
      for (int i = 0; i < H; ++i) us[i] = page_sum(prev[i]);
      if (grp == 0)
#pragma unroll
        for (int i = 0; i < H; ++i) s_up[j & 1][kh * H + i][rg][col] = us[i];
    };
    stream_stages<D, kNB>(p, bt, s_ring, 0, pe2, [&](int j, int slot) {
      if (j >= 2) flush(j - 2);
#pragma unroll
      for (int i = 0; i < H; ++i) page_logits<D, RTW>(qa, s_ring + (slot * S + kh * H + i) * PB, accs[slot][i]);
      sums_to_lds(j - 1, accs[slot ^ 1]);  // stage -1: zeros into the slot stage 1 fills before its flush
    });
    if (n1 >= 2) flush(n1 - 2);
    if (n1 >= 1) {
      if (n1 & 1) sums_to_lds(n1 - 1, accs[0]);
      else sums_to_lds(n1 - 1, accs[1]);
    }
    __syncthreads();
    if (n1 >= 1) flush(n1 - 1);
    __syncthreads();
  }
  // the remaining candidate pages one stage at a time (stage j = n1 + local)
  const int n_st2 = ceil_div_dev(cand_pages, S);
  stream_stages<D, kNB>(p, bt, s_ring, pe2, cand_pages, [&](int jl, int slot) {
    const int j = n1 + jl;
    if (jl > 0) flush(j - 1);
    f32x4_t acc[H][RTW];
#pragma unroll
    for (int i = 0; i < H; ++i) page_logits<D, RTW>(qa, s_ring + (slot * S + kh * H + i) * PB, acc[i]);
#pragma unroll
    for (int i = 0; i < H; ++i) {
      const int pg = j * S + kh * H + i;
      // H2O: the causal mask of the window keys (and of slots past the length)
      if (kAccum && pg >= p_full) causal_mask(acc[i], pg, -INFINITY);
      const float us = page_sum(acc[i]);
      if (grp == 0) s_up[j & 1][kh * H + i][rg][col] = us;  // pages past the candidates are never added
    }
  });
  if (n_st2 > n1) flush(n_st2 - 1);
  if (kAccum) return;  // the row block's partial u is written; h2o_chunk_apply_kernel adds the blocks
  __syncthreads();  // the unit's u is complete and visible to the work-group

  snapkv_pool(p, bt, L, n_lim, [&](int j) { return u[j]; }, s_ring, s_red);
}

template <int D, bool kAccum>
void launch_snapkv_d(const SnapParams& p, int num_units, int rows, hipStream_t stream) {
  const dim3 grid(num_units, p.n_rb);
  // H2O chunk scoring: one work-group per CU (grid = units x row blocks), the
  // pipelined stages and a deeper stream; SnapKV: two work-groups per CU, in
  // which the pipelined form would not fit the registers
  constexpr int occ = kAccum ? 2 : 4;
  constexpr bool pipe = kAccum;
  if (rows <= 64) {
    hipLaunchKernelGGL((snapkv_score_kernel<D, 1, kAccum, pipe, occ, kSnapRowGroups>), grid, dim3(kSnapThreads), 0,
                       stream, p);
  } else if constexpr (kAccum) {
    // 128 rows as two groups of 64: each key piece a wavefront reads from LDS
    // feeds four row tiles, which halves the LDS reads of a stage
    hipLaunchKernelGGL((snapkv_score_kernel<D, 4, kAccum, pipe, occ, 2>), grid, dim3(kSnapThreads), 0, stream, p);
  } else {
    hipLaunchKernelGGL((snapkv_score_kernel<D, 2, kAccum, pipe, occ, kSnapRowGroups>), grid, dim3(kSnapThreads), 0,
                       stream, p);
  }
}

// SnapKV with more than 128 scoring rows: the scoring kernel ran in its
// accumulate mode (row blocks of 128 rows, partial sums per block); this
// kernel adds the blocks' partials in block order and pools.  A unit the
// scoring kernel rejected (length or block table) is left alone.
__global__ __launch_bounds__(kSnapThreads) void snapkv_pool_kernel(const SnapParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t s_scr[(kSnapPoolChunk + 2 * kSnapHalo) * 8];
  __shared__ int s_red[kSnapWaves];
  const int unit = blockIdx.x;
  const int L = p.lengths[unit];
  if (L <= p.budget || L > p.max_len || L > p.max_pages * kPage || L > kSnapMaxPages * kPage) return;
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int n_pages = ceil_div_dev(L, kPage);
  int bad = 0;
  for (int i = threadIdx.x; i < n_pages; i += kSnapThreads) bad |= (bt[i] < 0 || (int64_t)bt[i] >= p.num_pages);
  if (block_reduce<kSnapThreads>(bad, s_red, [](int a, int b) { return a | b; })) return;
  const float* ub = p.u + (size_t)unit * p.n_rb * p.u_stride;
  snapkv_pool(p, bt, L, L - p.w, [&](int j) {
    float u = ub[j];
    for (int b = 1; b < p.n_rb; ++b) u += ub[(size_t)b * p.u_stride + j];
    return u;
  }, s_scr, s_red);
}

constexpr int kApplyThreads = 256;
constexpr int kApplySlots = 2048;  // slots per work-group

// H2O chunk scores: score(j) = (j in the chunk ? 0 : score(j)) + the row
// blocks' partial u (added in block order).  A unit the scoring kernel
// rejected (length or block table) is left alone.
__global__ __launch_bounds__(kApplyThreads) void h2o_chunk_apply_kernel(const SnapParams p) {
  __shared__ int s_red[kApplyThreads / kWave];
  const int unit = blockIdx.y;
  const int L = p.lengths[unit];
  if (L > p.max_len || L > p.max_pages * kPage || L > kSnapMaxPages * kPage || L < p.chunk) return;
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int n_pages = ceil_div_dev(L, kPage);
  int bad = 0;
  for (int i = threadIdx.x; i < n_pages; i += kApplyThreads) bad |= (bt[i] < 0 || (int64_t)bt[i] >= p.num_pages);
  if (block_reduce<kApplyThreads>(bad, s_red, [](int a, int b) { return a | b; })) return;
  // four consecutive slots per thread (one page holds them): 16-byte loads of
  // the partial rows and of the scores when the buffers are aligned
  const int j0 = blockIdx.x * kApplySlots;
  const int j1 = min(L, j0 + kApplySlots);
  const int cs = L - p.chunk;  // the chunk's first slot
  const float* ub = p.u + (size_t)unit * p.n_rb * p.u_stride;
  for (int j = j0 + 4 * (int)threadIdx.x; j < j1; j += 4 * kApplyThreads) {
    float* sc = p.score_pool + (size_t)bt[j >> 4] * kPage + (j & (kPage - 1));
    if (p.vec4 && j + 4 <= j1) {
      float4 u = *reinterpret_cast<const float4*>(ub + j);
      for (int b = 1; b < p.n_rb; ++b) {
        const float4 v = *reinterpret_cast<const float4*>(ub + (size_t)b * p.u_stride + j);
        u.x += v.x;
        u.y += v.y;
        u.z += v.z;
        u.w += v.w;
      }
      float4 o = *reinterpret_cast<const float4*>(sc);
      o.x = (j >= cs ? 0.f : o.x) + u.x;
      o.y = (j + 1 >= cs ? 0.f : o.y) + u.y;
      o.z = (j + 2 >= cs ? 0.f : o.z) + u.z;
      o.w = (j + 3 >= cs ? 0.f : o.w) + u.w;
      *reinterpret_cast<float4*>(sc) = o;
    } else {
      for (int t = j; t < min(j + 4, j1); ++t) {
        float u = ub[t];
        for (int b = 1; b < p.n_rb; ++b) u += ub[(size_t)b * p.u_stride + t];
        float* st = sc + (t - j);
        *st = (t >= cs ? 0.f : *st) + u;
      }
    }
  }
}


// ---------------------------------------------------------------- key split
// H2O chunk scoring with 257 .. 512 scoring rows (e.g. 128 queries x 4 heads):
// one work-group holds every row (eight wavefronts of 64 rows, four row tiles
// each) and a contiguous part of the unit's pages, and the unit's pages are
// split over gridDim.y work-groups.  Every wavefront reads every page of a
// stage from the ring (four pages, 64 MFMAs per wavefront between barriers,
// against 16 when a work-group holds a block of 128 rows and every key), and
// each page is staged once per unit instead of once per row block.  The row
// normalisers need every key, so the two passes are two kernels: the first
// leaves each part's (reference, sum) per row in the workspace, the second
// merges the parts in part order, forms each key's u over all the rows (the
// wavefronts' sums added in wavefront order) and writes the slot's new score
// (0 for the chunk's slots, plus u) itself.
constexpr int kSplitRows = 512;  // rows of a work-group
constexpr int kSplitThreads = 1024;
// row tiles of 16 rows per wavefront: 4 with 512 threads (two wavefronts per
// SIMD, up to 256 registers each), 2 with 1024 (four per SIMD, 128 registers)
template <int NT>
constexpr int kSplitRTW = kSplitRows / 16 / (NT / kWave);

// the pages [*pb, *pe) of part kp of nkp
__device__ __forceinline__ void key_part(int n_pages, int kp, int nkp, int* pb, int* pe) {
  *pb = (int)((int64_t)n_pages * kp / nkp);
  *pe = (int)((int64_t)n_pages * (kp + 1) / nkp);
}

// Unit checks shared by both passes (length, block table); the first pass's
// first part reports them.
template <int NT>
__device__ __forceinline__ bool split_unit_ok(const SnapParams& p, int unit, int L, bool report, int* s_red) {
  const int tid = threadIdx.x;
  if (L > p.max_len || L > p.max_pages * kPage || L > kSnapMaxPages * kPage || L < p.chunk) {
    if (report && tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return false;
  }
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int n_pages = ceil_div_dev(L, kPage);
  int bad = 0;
  for (int i = tid; i < n_pages; i += NT) bad |= (bt[i] < 0 || (int64_t)bt[i] >= p.num_pages);
  bad = block_reduce<NT>(bad, s_red, [](int a, int b) { return a | b; });
  if (bad) {
    if (report && tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
    return false;
  }
  return true;
}

// This wavefront's 16 * RTW query rows as A operands (rows past R are zero).
template <int D, int RTW>
__device__ __forceinline__ void split_queries(const SnapParams& p, int unit, int row0, uint4 (&qa)[RTW][D / 32]) {
  constexpr int KS = D / 32;
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane >> 4, col = lane & 15;
  const int req = unit / p.num_kv_heads, kvh = unit % p.num_kv_heads;
  const int G = p.q_per_kv, R = p.w * G, hq = p.num_kv_heads * G;
#pragma unroll
  for (int T = 0; T < RTW; ++T) {
    const int row = row0 + 16 * T + col;
    const int t = row / G, g = row - (row / G) * G;
    const uint16_t* src = p.q + (((size_t)req * p.w + t) * hq + (size_t)kvh * G + g) * D + 8 * grp;
#pragma unroll
    for (int k = 0; k < KS; ++k) qa[T][k] = row < R ? *reinterpret_cast<const uint4*>(src + 32 * k) : uint4{0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int k = 0; k < KS; ++k)
      asm volatile("" : "+v"(qa[T][k].x), "+v"(qa[T][k].y), "+v"(qa[T][k].z), "+v"(qa[T][k].w));
}

// The causal mask of a page holding window keys: key j is seen by the rows of
// window position t iff j <= L - w + t; padded rows see nothing.
template <int RTW>
__device__ __forceinline__ void split_mask(const SnapParams& p, f32x4_t (&a)[RTW], int pg, int L, int row0) {
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane >> 4, col = lane & 15;
  const int key = pg * kPage + col;
  const int G = p.q_per_kv, R = p.w * G;
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = row0 + 16 * T + 4 * grp + r;
      const int lim = row < R ? L - p.w + row / G : -1;
      if (key > lim) a[T][r] = -INFINITY;
    }
}

// Pass 1: per row, a lazy reference and the sum of exp2(c*z - reference) over
// this part's keys, merged over the 16 key lanes; norm[(unit * nkp + kp) *
// kSplitRows + row] = (reference, sum).
template <int D, int NT>
__global__ __launch_bounds__(NT, 2 * NT / kSnapThreads) void prefill_norm_kernel(const SnapParams p, float2* norm) {
  constexpr int RTW = kSplitRTW<NT>, S = kSnapStagePages, PB = 32 * D, NW = NT / kWave;
  __shared__ __attribute__((aligned(16))) uint8_t s_ring[2 * S * 32 * 128];
  __shared__ int s_red[NW];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int grp = lane >> 4, col = lane & 15;
  const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int unit = blockIdx.x, kp = blockIdx.y, nkp = gridDim.y;
  const int L = p.lengths[unit];
  if (!split_unit_ok<NT>(p, unit, L, kp == 0, s_red)) return;
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int n_pages = ceil_div_dev(L, kPage);
  int pb, pe;
  key_part(n_pages, kp, nkp, &pb, &pe);
  const int row0 = 16 * RTW * wv;
  uint4 qa[RTW][D / 32];
  split_queries<D, RTW>(p, unit, row0, qa);
  const float c = p.c;
  const int p_full = (L - p.w + 1) / kPage;  // pages below hold only keys every row sees
  float ref[RTW][4], sum[RTW][4];
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ref[T][r] = kRefInit;
      sum[T][r] = 0.f;
    }
  auto norm_page = [&](const f32x4_t(&a)[RTW]) {
    float dmax = -INFINITY;
    float d[RTW][4];
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        d[T][r] = fmaf(a[T][r], c, -ref[T][r]);
        dmax = fmaxf(dmax, d[T][r]);
      }
    if (__builtin_amdgcn_ballot_w64(dmax > kLazy) != 0) {
#pragma unroll
      for (int T = 0; T < RTW; ++T)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float zc = a[T][r] * c;
          const float m = fmaxf(ref[T][r], zc);
          sum[T][r] *= fast_exp2(ref[T][r] - m);
          d[T][r] = zc - m;
          ref[T][r] = m;
        }
    }
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) sum[T][r] += fast_exp2(d[T][r]);
  };
  stream_stages<D, 2 * kSnapBatches, NT>(p, bt, s_ring, pb, pe, [&](int j, int slot) {
    // page i + 1's MFMAs are issued before page i's exponentials
    f32x4_t acc[2][RTW];
    page_logits<D, RTW>(qa, s_ring + (slot * S) * PB, acc[0]);
#pragma unroll
    for (int i = 0; i < S; ++i) {
      if (i + 1 < S) page_logits<D, RTW>(qa, s_ring + (slot * S + i + 1) * PB, acc[(i + 1) & 1]);
      const int pg = pb + j * S + i;
      if (pg < pe) {
        if (pg >= p_full) split_mask<RTW>(p, acc[i & 1], pg, L, row0);
        norm_page(acc[i & 1]);
      }
    }
  });
  float2* out = norm + ((size_t)unit * nkp + kp) * kSplitRows;
#pragma unroll
  for (int T = 0; T < RTW; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int m = 1; m < 16; m <<= 1)
        merge_norm(ref[T][r], sum[T][r], shfl_xor_f(ref[T][r], m), shfl_xor_f(sum[T][r], m));
      if (col == 0) out[row0 + 16 * T + 4 * grp + r] = make_float2(ref[T][r], sum[T][r]);
    }
}

// Pass 2: bias = log2 of each row's softmax denominator (the parts merged in
// part order); u(j) = sum over every row of exp2(c*z - bias) for this part's
// keys; score(j) = (j in the chunk ? 0 : score(j)) + u(j).
template <int D, int NT>
__global__ __launch_bounds__(NT, 2 * NT / kSnapThreads) void prefill_score_kernel(const SnapParams p, const float2* norm) {
  constexpr int RTW = kSplitRTW<NT>, S = kSnapStagePages, PB = 32 * D, NW = NT / kWave;
  __shared__ __attribute__((aligned(16))) uint8_t s_ring[2 * S * 32 * 128];
  __shared__ float s_up[2][S][NW][kPage];  // [stage parity][page][wavefront][key]
  __shared__ int s_red[NW];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int grp = lane >> 4, col = lane & 15;
  const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int unit = blockIdx.x, kp = blockIdx.y, nkp = gridDim.y;
  const int L = p.lengths[unit];
  if (!split_unit_ok<NT>(p, unit, L, false, s_red)) return;
  const int32_t* bt = p.block_table + (size_t)unit * p.max_pages;
  const int n_pages = ceil_div_dev(L, kPage);
  int pb, pe;
  key_part(n_pages, kp, nkp, &pb, &pe);
  const int row0 = 16 * RTW * wv;
  const int R = p.w * p.q_per_kv;
  uint4 qa[RTW][D / 32];
  split_queries<D, RTW>(p, unit, row0, qa);
  const float c = p.c;
  const int p_full = (L - p.w + 1) / kPage;
  float bias[RTW][4];
  {
    const float2* nu = norm + (size_t)unit * nkp * kSplitRows;
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row0 + 16 * T + 4 * grp + r;
        float2 a = nu[row];
        for (int k = 1; k < nkp; ++k) {
          const float2 b = nu[(size_t)k * kSplitRows + row];
          merge_norm(a.x, a.y, b.x, b.y);
        }
        bias[T][r] = row < R ? a.x + __log2f(a.y) : INFINITY;
      }
  }
  // a page's weights summed over the lane's rows (a tree), then over the four
  // lane groups (rows 4*(lane/16)..+3 of each tile) of key lane%16
  auto page_sum = [&](const f32x4_t(&a)[RTW]) {
    float e[RTW * 4];
#pragma unroll
    for (int T = 0; T < RTW; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) e[4 * T + r] = fast_exp2(fmaf(a[T][r], c, -bias[T][r]));
#pragma unroll
    for (int n = RTW * 4; n > 1; n >>= 1)
#pragma unroll
      for (int k = 0; k < n / 2; ++k) e[k] = e[2 * k] + e[2 * k + 1];
    return lane_group_sum(e[0]);
  };
  // once stage j's barrier has passed, wavefront v < S adds the wavefronts'
  // sums of page v in wavefront order and writes the scores of its keys
  const int cs = L - p.chunk;  // the chunk's first slot
  auto flush = [&](int j) {
    if (wv < S && lane < kPage) {
      const int pg = pb + j * S + wv;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) v += s_up[j & 1][wv][w][lane];
      const int key = pg * kPage + lane;
      if (pg < pe && key < L) {
        float* sc = p.score_pool + (size_t)bt[pg] * kPage + lane;
        *sc = (key >= cs ? 0.f : *sc) + v;
      }
    }
  };
  const int n_st = ceil_div_dev(pe - pb, S);
  stream_stages<D, 2 * kSnapBatches, NT>(p, bt, s_ring, pb, pe, [&](int j, int slot) {
    if (j >= 1) flush(j - 1);
    f32x4_t acc[2][RTW];
    page_logits<D, RTW>(qa, s_ring + (slot * S) * PB, acc[0]);
#pragma unroll
    for (int i = 0; i < S; ++i) {
      if (i + 1 < S) page_logits<D, RTW>(qa, s_ring + (slot * S + i + 1) * PB, acc[(i + 1) & 1]);
      const int pg = pb + j * S + i;
      if (pg >= p_full) split_mask<RTW>(p, acc[i & 1], pg, L, row0);
      const float us = page_sum(acc[i & 1]);
      if (grp == 0) s_up[j & 1][i][wv][col] = us;  // pages past the part are never written out
    }
  });
  if (n_st >= 1) {
    __syncthreads();
    flush(n_st - 1);
  }
}

// The number of work-groups a unit's keys are split over: at least 256
// work-groups in all when the units allow, each over at least 8 pages.
static int prefill_key_parts(int32_t num_units, int32_t max_len) {
  const int64_t pages = ceil_div((int64_t)max_len, kPage);
  int64_t kp = ceil_div((int64_t)256, (int64_t)num_units);
  kp = std::min<int64_t>(kp, std::max<int64_t>(1, pages / 8));
  return (int)std::max<int64_t>(1, kp);
}

static bool prefill_key_split(int32_t q_per_kv, int32_t window) {
  const int64_t R = (int64_t)window * q_per_kv;
  return R > 2 * kPrefillBlockRows && R <= kSplitRows;
}

}  // namespace se

using namespace se;

// Workspace: the per-slot sums (one row per row block of 128 scoring rows),
// then (256-byte aligned) the eviction's deferred move lists, kMoveListInts
// ints per unit.  window = 0 sizes for at most 128 rows.
static int snapkv_row_blocks(int32_t q_per_kv, int32_t window) {
  const int64_t rows = (int64_t)window * q_per_kv;
  return rows > kSnapMaxRows ? (int)ceil_div(rows, kPrefillBlockRows) : 1;
}

static size_t snapkv_sums_bytes(int32_t num_units, int32_t max_len, int n_rb) {
  return align_up((size_t)num_units * n_rb * align_up((size_t)max_len, 64) * sizeof(float), 256);
}

size_t se_snapkv_workspace_bytes(int32_t num_units, int32_t max_len, int32_t q_per_kv, int32_t window) {
  if (num_units <= 0 || max_len <= 0) return 0;
  return snapkv_sums_bytes(num_units, max_len, snapkv_row_blocks(q_per_kv, window)) +
         (size_t)num_units * kMoveListInts * sizeof(int32_t);
}

extern "C" se_status se_snapkv_compact(const se_kv_view* kv, int32_t q_per_kv, const void* q_obs,
                                       int32_t window, int32_t kernel, float scale, int32_t budget,
                                       int32_t max_len, uint32_t flags, int32_t* freed_pages,
                                       int32_t freed_stride, int32_t* freed_count, void* ws,
                                       size_t ws_bytes, int32_t* dev_err, hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->kv_pool == nullptr || kv->pos_pool == nullptr || kv->score_pool == nullptr ||
      q_obs == nullptr || dev_err == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if ((flags & ~SE_SNAPKV_SCORE_ONLY) != 0) return SE_ERR_INVALID_ARGUMENT;
  if (q_per_kv < 1 || window < 1 || budget < window || max_len < 1) return SE_ERR_INVALID_ARGUMENT;
  if (kernel < 1 || (kernel & 1) == 0) return SE_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !(scale < INFINITY)) return SE_ERR_INVALID_ARGUMENT;
  if (freed_pages != nullptr && freed_stride < kv->max_pages) return SE_ERR_INVALID_ARGUMENT;
  if ((int64_t)window * q_per_kv > 8 * kSnapMaxRows || kernel / 2 > kSnapMaxHalf) return SE_ERR_UNSUPPORTED;
  if (budget > kMaxBudget || max_len > kSnapMaxPages * kPage) return SE_ERR_UNSUPPORTED;
  const int n_rb = snapkv_row_blocks(q_per_kv, window);
  const size_t need = se_snapkv_workspace_bytes(kv->num_units, max_len, q_per_kv, window);
  if (ws == nullptr || ws_bytes < need) return SE_ERR_WORKSPACE;

  SnapParams p;
  p.kv = static_cast<const uint16_t*>(kv->kv_pool);
  p.pos_pool = kv->pos_pool;
  p.score_pool = kv->score_pool;
  p.block_table = kv->block_table;
  p.lengths = kv->lengths;
  p.q = static_cast<const uint16_t*>(q_obs);
  p.u = static_cast<float*>(ws);
  p.num_pages = kv->num_pages;
  p.max_pages = kv->max_pages;
  p.num_kv_heads = kv->num_kv_heads;
  p.q_per_kv = q_per_kv;
  p.w = window;
  p.half = kernel / 2;
  p.budget = budget;
  p.max_len = max_len;
  p.u_stride = (int32_t)align_up((size_t)max_len, 64);
  p.c = scale * kLog2e;
  p.dev_err = dev_err;
  const int rows = window * q_per_kv;
  p.n_rb = n_rb;
  p.chunk = 0;
  p.vec4 = 0;
  p.snap_wide = n_rb > 1;
  if (n_rb == 1) {  // one work-group per unit scores and pools
    if (kv->head_dim == 128)
      launch_snapkv_d<128, false>(p, kv->num_units, rows, stream);
    else
      launch_snapkv_d<64, false>(p, kv->num_units, rows, stream);
  } else {  // row blocks of 128 rows score every key, then the pool kernel adds them
    if (kv->head_dim == 128)
      launch_snapkv_d<128, true>(p, kv->num_units, kPrefillBlockRows, stream);
    else
      launch_snapkv_d<64, true>(p, kv->num_units, kPrefillBlockRows, stream);
    hipLaunchKernelGGL(snapkv_pool_kernel, dim3(kv->num_units), dim3(kSnapThreads), 0, stream, p);
  }
  st = launch_status();
  if (st != SE_OK || (flags & SE_SNAPKV_SCORE_ONLY)) return st;

  EvictParams e;
  e.kv = static_cast<uint16_t*>(kv->kv_pool);
  e.pos_pool = kv->pos_pool;
  e.score_pool = kv->score_pool;
  e.block_table = kv->block_table;
  e.lengths = kv->lengths;
  e.num_pages = kv->num_pages;
  e.max_pages = kv->max_pages;
  e.budget = budget;
  e.recent = window;
  e.max_len = max_len;
  e.freed_pages = freed_pages;
  e.freed_stride = freed_stride;
  e.freed_count = freed_count;
  e.dev_err = dev_err;
  e.moves = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + snapkv_sums_bytes(kv->num_units, max_len, n_rb));
  launch_evict(e, kv->num_units, kv->head_dim, stream);
  return launch_status();
}

// Workspace: the row blocks' partial sums (or, with the keys split, each
// part's row normalisers), then the eviction's move lists.
static size_t prefill_sums_bytes(int32_t num_units, int32_t max_len, int32_t q_per_kv, int32_t window) {
  if (prefill_key_split(q_per_kv, window))
    return align_up((size_t)num_units * prefill_key_parts(num_units, max_len) * kSplitRows * sizeof(float2), 256);
  const size_t n_rb = (size_t)ceil_div((int64_t)window * q_per_kv, kPrefillBlockRows);
  return align_up((size_t)num_units * n_rb * align_up((size_t)max_len, 64) * sizeof(float), 256);
}

size_t se_h2o_prefill_workspace_bytes(int32_t num_units, int32_t max_len, int32_t q_per_kv, int32_t window) {
  if (num_units <= 0 || max_len <= 0 || q_per_kv <= 0 || window <= 0) return 0;
  return prefill_sums_bytes(num_units, max_len, q_per_kv, window) +
         (size_t)num_units * kMoveListInts * sizeof(int32_t);
}

extern "C" se_status se_h2o_prefill_chunk(const se_kv_view* kv, int32_t q_per_kv, const void* q_score,
                                          int32_t score_window, int32_t chunk_len, float scale, int32_t budget,
                                          int32_t recent, int32_t max_len, int32_t* freed_pages,
                                          int32_t freed_stride, int32_t* freed_count, void* ws, size_t ws_bytes,
                                          int32_t* dev_err, hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (kv->kv_pool == nullptr || kv->pos_pool == nullptr || kv->score_pool == nullptr || q_score == nullptr ||
      dev_err == nullptr)
    return SE_ERR_INVALID_ARGUMENT;
  if (q_per_kv < 1 || score_window < 1 || chunk_len < score_window || budget < 1 || recent < 0 || max_len < 1)
    return SE_ERR_INVALID_ARGUMENT;
  if (!(scale > 0.f) || !(scale < INFINITY)) return SE_ERR_INVALID_ARGUMENT;
  if (freed_pages != nullptr && freed_stride < kv->max_pages) return SE_ERR_INVALID_ARGUMENT;
  if ((int64_t)score_window * q_per_kv > 8 * kSnapMaxRows) return SE_ERR_UNSUPPORTED;
  // a budget of at least max_len evicts nothing, so it needs no eviction capacity
  if ((budget > kMaxBudget && budget < max_len) || max_len > kSnapMaxPages * kPage) return SE_ERR_UNSUPPORTED;
  if (ws == nullptr || ws_bytes < se_h2o_prefill_workspace_bytes(kv->num_units, max_len, q_per_kv, score_window))
    return SE_ERR_WORKSPACE;

  SnapParams p;
  p.kv = static_cast<const uint16_t*>(kv->kv_pool);
  p.pos_pool = kv->pos_pool;
  p.score_pool = kv->score_pool;
  p.block_table = kv->block_table;
  p.lengths = kv->lengths;
  p.q = static_cast<const uint16_t*>(q_score);
  p.u = static_cast<float*>(ws);
  p.num_pages = kv->num_pages;
  p.max_pages = kv->max_pages;
  p.num_kv_heads = kv->num_kv_heads;
  p.q_per_kv = q_per_kv;
  p.w = score_window;
  p.half = 0;
  p.budget = budget;
  p.max_len = max_len;
  p.u_stride = (int32_t)align_up((size_t)max_len, 64);
  p.n_rb = (int32_t)ceil_div((int64_t)score_window * q_per_kv, kPrefillBlockRows);
  p.chunk = chunk_len;
  p.snap_wide = 0;
  p.vec4 = (reinterpret_cast<uintptr_t>(kv->score_pool) % 16 == 0 && reinterpret_cast<uintptr_t>(ws) % 16 == 0) ? 1 : 0;
  p.c = scale * kLog2e;
  p.dev_err = dev_err;
  if (prefill_key_split(q_per_kv, score_window)) {
    // every row in one work-group, the unit's pages split over several
    const dim3 grid(kv->num_units, prefill_key_parts(kv->num_units, max_len));
    float2* norm = static_cast<float2*>(ws);
    // head_dim 128: 1024 threads (a stage is one 16-byte piece per thread);
    // 64: 512
    if (kv->head_dim == 128) {
      hipLaunchKernelGGL((prefill_norm_kernel<128, kSplitThreads>), grid, dim3(kSplitThreads), 0, stream, p, norm);
      hipLaunchKernelGGL((prefill_score_kernel<128, kSplitThreads>), grid, dim3(kSplitThreads), 0, stream, p, norm);
    } else {
      hipLaunchKernelGGL((prefill_norm_kernel<64, kSnapThreads>), grid, dim3(kSnapThreads), 0, stream, p, norm);
      hipLaunchKernelGGL((prefill_score_kernel<64, kSnapThreads>), grid, dim3(kSnapThreads), 0, stream, p, norm);
    }
  } else {
    const int rows = std::min(score_window * q_per_kv, kPrefillBlockRows);
    if (kv->head_dim == 128)
      launch_snapkv_d<128, true>(p, kv->num_units, rows, stream);
    else
      launch_snapkv_d<64, true>(p, kv->num_units, rows, stream);
    hipLaunchKernelGGL(h2o_chunk_apply_kernel, dim3((unsigned)ceil_div(max_len, kApplySlots), kv->num_units),
                       dim3(kApplyThreads), 0, stream, p);
  }
  st = launch_status();
  if (st != SE_OK) return st;

  EvictParams e;
  e.kv = static_cast<uint16_t*>(kv->kv_pool);
  e.pos_pool = kv->pos_pool;
  e.score_pool = kv->score_pool;
  e.block_table = kv->block_table;
  e.lengths = kv->lengths;
  e.num_pages = kv->num_pages;
  e.max_pages = kv->max_pages;
  e.budget = budget;
  e.recent = recent;
  e.max_len = max_len;
  e.freed_pages = freed_pages;
  e.freed_stride = freed_stride;
  e.freed_count = freed_count;
  e.dev_err = dev_err;
  e.moves = reinterpret_cast<int32_t*>(static_cast<char*>(ws) +
                                       prefill_sums_bytes(kv->num_units, max_len, q_per_kv, score_window));
  launch_evict(e, kv->num_units, kv->head_dim, stream);
  return launch_status();
}
