// se_decode_attend: append the decode token, split-K paged GQA decode attention
// over a per-unit view, and the fused H2O score update.
//
// Math (Appendix A.1, eq. background-selected-attention; Appendix A.3, eq.
// background-h2o-score): for each query row a of a unit, z_j = scale * <q_a, k_j>
// over the read set, out_a = sum_j softmax(z)_j v_j, and with accumulation every
// read slot's score grows by its weight summed over the unit's G rows.
//
// Work decomposition.  A unit's visited pages are cut into n_split ranges; one
// 256-thread work-group (four wavefronts) streams one range, each wavefront one
// page at a time:
//   * QK layout: lane = 4*r + j reads row r, columns [j*D/4, (j+1)*D/4) of the
//     page's K block with 16-byte loads, forms bf16 pair dot products with the
//     G query rows (v_dot2c_f32_bf16), and a quad DPP reduction gives every lane
//     of the quad the G logits of row r; lane j keeps head j.
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
#include "se_common.h"

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
  int32_t* dev_err;
};

struct AttendWs {
  size_t part, pbuf, mref, total;
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
__device__ void finish_unit(const AttendParams& p, const UnitGeom& g, const float* fin_m,
                            const float* fin_il) {
  const size_t ubase_p = (size_t)g.unit * p.n_visit_max;
  if (p.accumulate) {
    for (int idx = threadIdx.x; idx < g.n_visit * kPage; idx += blockDim.x) {
      const int vp = idx >> 4;
      const int rr = idx & (kPage - 1);
      int lp = vp;
      if (g.quest) {
        lp = vp < p.top_k ? p.sel[(size_t)g.unit * p.top_k + vp] : g.cur_page;
        if (lp < 0 || (vp < p.top_k && lp >= g.cur_page)) continue;
      }
      const int slot = lp * kPage + rr;
      if (slot >= g.Lp) continue;
      const int phys = p.block_table[(size_t)g.unit * p.max_pages + lp];
      if (phys < 0 || (int64_t)phys >= p.num_pages) continue;
      float a = 0.f;
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float w = p.pbuf[((ubase_p + vp) * kPage + rr) * G + h];
        const float mr = p.mref[(ubase_p + vp) * G + h];
        a += w * fast_exp2(mr - fin_m[h]) * fin_il[h];
      }
      float* up = p.score_pool + (size_t)phys * kPage + rr;
      *up = (g.append && slot == g.L) ? a : *up + a;
    }
  }
  if (g.append && threadIdx.x == 0) p.lengths[g.unit] = g.Lp;
}

template <int D, int G>
__global__ __launch_bounds__(256) void decode_attend_kernel(const AttendParams p) {
  constexpr int NW = 4;            // wavefronts per work-group
  constexpr int QC = D / 4;        // K columns per lane (QK layout)
  constexpr int QW = QC / 2;       // bf16 pairs per lane per head
  constexpr int K4 = QC / 8;       // 16-byte loads per lane per K row chunk
  constexpr int RS = 128 / D;      // row sets of the PV layout
  constexpr int RPL = kPage / RS;  // rows per lane (PV layout)
  constexpr int HP = D / 2;        // lanes per row set (two columns each)
  constexpr float kBump = 8.0f;    // rescale only when a logit beats the reference by 2^8

  __shared__ float lds_p[NW][kPage * G];
  __shared__ float lds_m[NW][G];
  __shared__ float lds_l[NW][G];
  __shared__ float lds_o[NW][G][D];
  __shared__ float fin_m[G];
  __shared__ float fin_il[G];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int unit = blockIdx.x / p.n_split;
  const int split = blockIdx.x - unit * p.n_split;
  const UnitGeom g = unit_geom(p, unit);
  const int req = g.req, kvh = g.kvh, L = g.L, Lp = g.Lp, cur_page = g.cur_page, n_visit = g.n_visit;
  const bool append = g.append, quest = g.quest, bad = g.bad;
  const int Hq = p.hkv * G;
  const int vbeg = split * p.pps;
  const int vend = min(vbeg + p.pps, n_visit);

  const size_t ubase_p = (size_t)unit * p.n_visit_max;  // page-indexed workspace rows

  // QK-layout coordinates.
  const int r = lane >> 2;
  const int j = lane & 3;
  // PV-layout coordinates.
  const int col = 2 * (lane % HP);
  const int rs = lane / HP;

  uint32_t qreg[G][QW];
  {
    const uint16_t* qb = p.q + ((size_t)req * Hq + (size_t)kvh * G) * D + j * QC;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const uint4* src = reinterpret_cast<const uint4*>(qb + (size_t)h * D);
#pragma unroll
      for (int i = 0; i < K4; ++i) {
        uint4 t = src[i];
        qreg[h][4 * i + 0] = t.x;
        qreg[h][4 * i + 1] = t.y;
        qreg[h][4 * i + 2] = t.z;
        qreg[h][4 * i + 3] = t.w;
      }
    }
  }

  float m_ref[G];
  float o_acc[G][2];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_ref[h] = -INFINITY;
    o_acc[h][0] = 0.f;
    o_acc[h][1] = 0.f;
  }
  float l_own = 0.f;

  const uint16_t* knew_row =
      append ? p.k_new + ((size_t)req * p.hkv + kvh) * D : nullptr;
  const uint16_t* vnew_row =
      append ? p.v_new + ((size_t)req * p.hkv + kvh) * D : nullptr;

  for (int vp = vbeg + wave; vp < vend; vp += NW) {
    int lp;
    if (quest) {
      lp = vp < p.top_k ? p.sel[(size_t)unit * p.top_k + vp] : cur_page;
      if (lp < 0) continue;
      if (vp < p.top_k && lp >= cur_page) {
        if (lane == 0) set_error(p.dev_err, SE_DEVERR_BAD_SELECTION);
        continue;
      }
    } else {
      lp = vp;
    }
    const int phys = p.block_table[(size_t)unit * p.max_pages + lp];
    if (phys < 0 || (int64_t)phys >= p.num_pages) {
      if (lane == 0) set_error(p.dev_err, SE_DEVERR_BAD_PAGE);
      continue;
    }
    const int row0 = lp * kPage;
    const int nrows = min(kPage, Lp - row0);
    const bool has_new = append && L >= row0 && L < row0 + kPage;
    const int rn = L - row0;
    const uint16_t* kpage = p.kv + (size_t)phys * (2 * kPage * D);
    const uint16_t* vpage = kpage + kPage * D;

    // ---- loads: K chunk (QK layout) and V column pairs (PV layout)
    const int rk = min(r, nrows - 1);
    const uint16_t* krow = (has_new && rk == rn) ? knew_row : kpage + rk * D;
    uint4 kreg[K4];
#pragma unroll
    for (int i = 0; i < K4; ++i) kreg[i] = reinterpret_cast<const uint4*>(krow + j * QC)[i];
    uint32_t vreg[RPL];
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      const int rv = min(rs * RPL + i, nrows - 1);
      const uint16_t* vrow = (has_new && rv == rn) ? vnew_row : vpage + rv * D;
      vreg[i] = *reinterpret_cast<const uint32_t*>(vrow + col);
    }

    // ---- append: the new token's row enters the pool
    if (has_new) {
      uint16_t* kdst = const_cast<uint16_t*>(kpage) + rn * D;
      if (r == rn) {
#pragma unroll
        for (int i = 0; i < K4; ++i) reinterpret_cast<uint4*>(kdst + j * QC)[i] = kreg[i];
        if (p.meta_pool != nullptr) {
          uint16_t* mn = p.meta_pool + (size_t)phys * 2 * D + j * QC;
          uint16_t* mx = mn + D;
          const uint16_t* kn = knew_row + j * QC;
          for (int c = 0; c < QC; ++c) {
            const uint16_t kb = kn[c];
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
      }
      if (rn >= rs * RPL && rn < (rs + 1) * RPL)
        *reinterpret_cast<uint32_t*>(const_cast<uint16_t*>(vpage) + rn * D + col) = vreg[rn - rs * RPL];
      if (lane == 0) {
        p.pos_pool[(size_t)phys * kPage + rn] = p.new_pos[req];
        if (p.score_pool != nullptr) p.score_pool[(size_t)phys * kPage + rn] = 0.f;
      }
    }

    // ---- logits of row r for all G heads, reduced over the quad
    float acc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = 0.f;
#pragma unroll
    for (int i = 0; i < K4; ++i) {
      const uint32_t kw[4] = {kreg[i].x, kreg[i].y, kreg[i].z, kreg[i].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = dot2bf16(qreg[h][4 * i + e], kw[e], acc[h]);
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) acc[h] = quad_sum(acc[h]);
    float z = acc[0];
#pragma unroll
    for (int h = 1; h < G; ++h) z = (j == h) ? acc[h] : z;
    const bool valid = (r < nrows) && (j < G);
    const float z2 = valid ? z * p.scale_log2 : -INFINITY;
    if (p.logits != nullptr && valid)
      p.logits[((size_t)unit * G + j) * p.logits_stride + row0 + r] = z * p.scale;

    // ---- reference maximum: raised only when some logit beats it by 2^kBump
    float mown = m_ref[0];
#pragma unroll
    for (int h = 1; h < G; ++h) mown = (j == h) ? m_ref[h] : mown;
    const bool need = valid && (z2 > mown + kBump);
    if (__ballot(need) != 0) {
      float mx = z2;
      mx = fmaxf(mx, shfl_xor_f(mx, 4));
      mx = fmaxf(mx, shfl_xor_f(mx, 8));
      mx = fmaxf(mx, shfl_xor_f(mx, 16));
      mx = fmaxf(mx, shfl_xor_f(mx, 32));
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float mh = fmaxf(m_ref[h], __shfl(mx, h, kWave));
        const float f = fast_exp2(m_ref[h] - mh);
        o_acc[h][0] *= f;
        o_acc[h][1] *= f;
        if (j == h) l_own *= f;
        m_ref[h] = mh;
      }
      mown = m_ref[0];
#pragma unroll
      for (int h = 1; h < G; ++h) mown = (j == h) ? m_ref[h] : mown;
    }
    const float pj = valid ? fast_exp2(z2 - mown) : 0.f;
    l_own += pj;
    if (p.accumulate) {
      if (j < G) p.pbuf[((ubase_p + vp) * kPage + r) * G + j] = pj;
      if (lane < G) {
        float mv = m_ref[0];
#pragma unroll
        for (int h = 1; h < G; ++h) mv = (lane == h) ? m_ref[h] : mv;
        p.mref[(ubase_p + vp) * G + lane] = mv;
      }
    }

    // ---- PV: broadcast the page's weights through LDS
    if (j < G) lds_p[wave][r * G + j] = pj;
    wave_lds_sync();
#pragma unroll
    for (int i = 0; i < RPL; ++i) {
      const int rr = rs * RPL + i;
      const float v0 = bf16lo(vreg[i]);
      const float v1 = bf16hi(vreg[i]);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float ph = lds_p[wave][rr * G + h];
        o_acc[h][0] = fmaf(ph, v0, o_acc[h][0]);
        o_acc[h][1] = fmaf(ph, v1, o_acc[h][1]);
      }
    }
    wave_lds_sync();
  }

  // ---- per-wavefront totals into LDS
  float lsum = l_own;
  lsum += shfl_xor_f(lsum, 4);
  lsum += shfl_xor_f(lsum, 8);
  lsum += shfl_xor_f(lsum, 16);
  lsum += shfl_xor_f(lsum, 32);
  if (RS == 2) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      o_acc[h][0] += shfl_xor_f(o_acc[h][0], 32);
      o_acc[h][1] += shfl_xor_f(o_acc[h][1], 32);
    }
  }
  if (lane < G) {
    float mv = m_ref[0];
#pragma unroll
    for (int h = 1; h < G; ++h) mv = (lane == h) ? m_ref[h] : mv;
    lds_m[wave][lane] = mv;
    lds_l[wave][lane] = lsum;
  }
  if (lane < HP) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      lds_o[wave][h][col] = o_acc[h][0];
      lds_o[wave][h][col + 1] = o_acc[h][1];
    }
  }
  __syncthreads();

  // ---- work-group partial (fixed wavefront order)
  const bool single = p.n_split == 1;
  float* part_u = p.part + (size_t)unit * p.n_split * G * (D + 2);
  for (int idx = tid; idx < G * D; idx += 256) {
    const int h = idx / D;
    const int c = idx - h * D;
    float ms = lds_m[0][h];
#pragma unroll
    for (int w = 1; w < NW; ++w) ms = fmaxf(ms, lds_m[w][h]);
    float o = 0.f, l = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = lds_m[w][h] == -INFINITY ? 0.f : fast_exp2(lds_m[w][h] - ms);
      o += lds_o[w][h][c] * f;
      l += lds_l[w][h] * f;
    }
    if (single) {
      if (!bad) {
        p.out[((size_t)req * Hq + kvh * G + h) * D + c] = o / l;
        if (c == 0) {
          if (p.lse != nullptr) p.lse[(size_t)req * Hq + kvh * G + h] = (ms + __log2f(l)) * kLn2;
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

  if (!single) return;  // the combine kernel finishes the unit
  __syncthreads();
  if (bad) {
    if (tid == 0) set_error(p.dev_err, SE_DEVERR_BAD_LENGTH);
    return;
  }
  finish_unit<G>(p, g, fin_m, fin_il);
}

// Second pass when a unit is split over several work-groups: combines the
// partials (m, l, o) in split order, writes out and lse, then finishes the unit.
template <int D, int G>
__global__ __launch_bounds__(256) void decode_combine_kernel(const AttendParams p) {
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
  finish_unit<G>(p, g, fin_m, fin_il);
}

template <int D, int G>
static void launch_attend(const AttendParams& prm, int grid, hipStream_t stream) {
  hipLaunchKernelGGL((decode_attend_kernel<D, G>), dim3(grid), dim3(256), 0, stream, prm);
  if (prm.n_split > 1)
    hipLaunchKernelGGL((decode_combine_kernel<D, G>), dim3(grid / prm.n_split), dim3(256), 0, stream,
                       prm);
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

extern "C" se_status se_decode_attend(const se_kv_view* kv, int32_t q_per_kv, const void* q,
                                      const void* k_new, const void* v_new,
                                      const int32_t* new_pos, const int32_t* sel_pages,
                                      int32_t top_k, float scale, int32_t max_len,
                                      uint32_t flags, float* out, float* lse, float* logits,
                                      int32_t logits_stride, void* ws, size_t ws_bytes,
                                      int32_t* dev_err, hipStream_t stream) {
  se_status st = check_view(kv);
  if (st != SE_OK) return st;
  if (q_per_kv != 1 && q_per_kv != 2 && q_per_kv != 4) return SE_ERR_UNSUPPORTED;
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
  const SplitShape s = split_shape(kv->num_units, attend_n_visit(max_len, kv->max_pages, top_k));
  const AttendWs lay = attend_ws_layout(kv->num_units, s, q_per_kv, D);
  if (ws == nullptr || ws_bytes < lay.total) return SE_ERR_WORKSPACE;

  AttendParams prm;
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
  prm.dev_err = dev_err;

  const int64_t grid = (int64_t)kv->num_units * s.n_split;
  if (grid > INT32_MAX) return SE_ERR_UNSUPPORTED;
  if (D == 128) {
    if (q_per_kv == 4) launch_attend<128, 4>(prm, (int)grid, stream);
    else if (q_per_kv == 2) launch_attend<128, 2>(prm, (int)grid, stream);
    else launch_attend<128, 1>(prm, (int)grid, stream);
  } else {
    if (q_per_kv == 4) launch_attend<64, 4>(prm, (int)grid, stream);
    else if (q_per_kv == 2) launch_attend<64, 2>(prm, (int)grid, stream);
    else launch_attend<64, 1>(prm, (int)grid, stream);
  }
  return launch_status();
}
