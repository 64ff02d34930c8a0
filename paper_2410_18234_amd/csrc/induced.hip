// Induced distribution r of the importance-weighted selection (step 1 of the
// canonical decomposition, Theorem 1), K = 2 and K = 3 i.i.d. drafts, gfx950.
//
// Notation: p = target, q = draft, w = p / q.  With the classical weights
// (index probability proportional to w, stated after Definition 1), the
// marginal of the selected token (proof of Theorem 1) is, by exchangeability
// of the drafts,
//   K = 2: r(y) = 2 p(y) S(y),  S(y) = sum_{x in supp} q(x) / (w(y) + w(x))
//          (the pair form eq. p_Ieq0 with w_{k,i} = w(k)/(w(k)+w(i)));
//   K = 3: r(y) = 3 p(y) sum_{x2,x3 in supp} q(x2) q(x3) / (w(y) + w(x2) + w(x3));
//   r(y) = q(y) Q0^(K-1) when p(y) = 0 < q(y), and 0 when q(y) = 0.
//
// Both sums are Stieltjes sums sum_m c_m / (a + s_m) of a query a = w(y) over
// the "poles" (s_m, c_m).  A reciprocal costs about three FMA issue slots on
// gfx950, so poles are grouped in chunks of C (4 or 8) and a chunk is
// evaluated as one rational function N(a) / D(a):
//   D(a) = prod_c (a + s_c),   N(a) = sum_c c_c prod_{c' != c} (a + s_c'),
// by Horner: 2C - 1 FMAs + 1 add + 1 reciprocal + 1 FMA per (query, chunk)
// instead of C adds + C reciprocals + C FMAs.  All coefficients and the
// argument are non-negative, so Horner has no cancellation; the weights are
// scaled by a power of two per row (w' = w 2^s) so that D stays inside the
// fp32 range, and rows whose weight range is too wide for that use one
// reciprocal per pair.  Sums are accumulated in fp32 over one LDS tile
// (<= 256 terms) and folded into fp64.
#include "common.h"

#include <math.h>

#include <algorithm>

namespace mdss {

namespace {

constexpr int kPrepThreads = 1024;
constexpr int kSweepThreads = 256;
constexpr int kTileFloats = 2048;  // pole-stream floats per LDS tile (8 KB)
constexpr int kRat8MaxRange = 28;  // binary exponent range of the weights allowed for 8-pole chunks
constexpr int kRat4MaxRange = 56;  // ... for 4-pole chunks
constexpr int kBlockPolesPrep = 128;  // K = 2 rows are padded to whole 128-pole blocks
#ifndef MDSS_MFMA_MT
#define MDSS_MFMA_MT 4
#endif
#ifndef MDSS_MFMA_NW
#define MDSS_MFMA_NW 4
#endif

__host__ __device__ inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

__device__ inline int mode_chunk(int mode) { return mode == kRat8 ? 8 : (mode == kRat4 ? 4 : 1); }

// ------------------------------------------------------------------ preparation
// One workgroup per row: validate the row, count the support, find the draft
// mass Q0 of zero-weight tokens and the weight range, choose the evaluation
// mode and scale, compact the support (ascending token id) into the workspace
// and write r for every token outside the support (and for flagged rows).
__global__ __launch_bounds__(kPrepThreads) void prep_kernel(const float* __restrict__ p, const float* __restrict__ q,
                                                             int64_t V, int K, int s_max, float* __restrict__ r,
                                                             int32_t* __restrict__ row_status, Workspace ws) {
  const int64_t b = blockIdx.x;
  const float* pb = p + b * V;
  const float* qb = q + b * V;
  float* rb = r + b * V;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int kWaves = kPrepThreads / 64;
  __shared__ double s_q0[kWaves];
  __shared__ int s_cnt[kWaves], s_cnt_pos[kWaves], s_bad[kWaves];
  __shared__ float s_wmin[kWaves], s_wmax[kWaves];
  __shared__ int s_scan[kWaves];
  __shared__ RowHdr s_hdr;

  int bad = 0, cnt = 0, cnt_pos = 0;
  double q0 = 0.0;
  float wmin = INFINITY, wmax = 0.0f;
  for (int64_t x = tid; x < V; x += kPrepThreads) {
    const float pv = pb[x], qv = qb[x];
    bad |= (int)bad_prob(pv) | (int)bad_prob(qv);
    if (qv > 0.0f) {
      ++cnt;
      cnt_pos += pv > 0.0f;
      if (pv == 0.0f) {
        q0 += (double)qv;
      } else {
        const float w = pv / qv;
        wmin = fminf(wmin, w);
        wmax = fmaxf(wmax, w);
      }
    }
  }
  bad = wave_sum_int(bad);
  cnt = wave_sum_int(cnt);
  cnt_pos = wave_sum_int(cnt_pos);
  q0 = wave_sum(q0);
  wmin = wave_min(wmin);
  wmax = wave_max(wmax);
  if (lane == 0) {
    s_bad[wid] = bad;
    s_cnt[wid] = cnt;
    s_cnt_pos[wid] = cnt_pos;
    s_q0[wid] = q0;
    s_wmin[wid] = wmin;
    s_wmax[wid] = wmax;
  }
  __syncthreads();
  if (tid == 0) {
    int tb = 0, tc = 0, tp = 0;
    double tq = 0.0;
    float mn = INFINITY, mx = 0.0f;
    for (int i = 0; i < kWaves; ++i) {
      tb |= s_bad[i];
      tc += s_cnt[i];
      tp += s_cnt_pos[i];
      tq += s_q0[i];
      mn = fminf(mn, s_wmin[i]);
      mx = fmaxf(mx, s_wmax[i]);
    }
    RowHdr h;
    // K = 2 compacts the positive-weight tokens only (a zero-weight pole adds q(y) Q0 in closed form);
    // K = 3 keeps the whole support as poles
    h.n = K == 2 ? tp : tc;
    h.q0 = tq;
    h.pad = 0.0;
    h.scale = 0;
    h.flags = tb ? kRowBadProb : ((K == 3 && tc > s_max) ? kRowSupport : 0);
    if (h.flags || tc == 0 || !(mx > 0.0f)) {
      h.mode = kSkip;  // flagged, empty support, or every weight zero
    } else {
      int e_lo, e_hi;
      frexpf(mn, &e_lo);
      frexpf(mx, &e_hi);
      const int range = e_hi - e_lo;
      if (!isfinite(mx) || range > kRat4MaxRange) {
        h.mode = kDirect;
      } else {
        h.mode = range <= kRat8MaxRange ? kRat8 : kRat4;
        h.scale = -((e_lo + e_hi) >> 1);
      }
    }
    s_hdr = h;
    ws.hdr[b] = h;
    if (row_status && h.flags) row_status[b] |= h.flags;
  }
  __syncthreads();
  const RowHdr h = s_hdr;
  if (h.flags) {
    for (int64_t x = tid; x < V; x += kPrepThreads) rb[x] = NAN;
    return;
  }
  const bool all_zero_weight = (h.mode == kSkip);  // support non-empty but every w == 0, or empty support
  const double zero_w_factor = (K == 2) ? h.q0 : h.q0 * h.q0;

  int32_t* idx = ws.idx + b * ws.Sp;
  float* wc = ws.wc + b * ws.Sp;
  float* qc = ws.qc + b * ws.Sp;
  int running = 0;
  for (int64_t base = 0; base < V; base += 4 * kPrepThreads) {
    const int64_t x0 = base + 4 * (int64_t)tid;
    float pv[4], qv[4];
    int c = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t x = x0 + i;
      pv[i] = (x < V) ? pb[x] : 0.0f;
      qv[i] = (x < V) ? qb[x] : 0.0f;
      c += (qv[i] > 0.0f) && (K != 2 || pv[i] > 0.0f);
    }
    const int incl = wave_inclusive_scan_int(c, lane);
    if (lane == 63) s_scan[wid] = incl;
    __syncthreads();
    int wave_off = 0, total = 0;
    for (int i = 0; i < kWaves; ++i) {
      wave_off += (i < wid) ? s_scan[i] : 0;
      total += s_scan[i];
    }
    int off = running + wave_off + incl - c;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t x = x0 + i;
      if (x >= V) break;
      if (qv[i] > 0.0f) {
        if (all_zero_weight || (K == 2 && !(pv[i] > 0.0f))) {
          rb[x] = (float)((double)qv[i] * zero_w_factor);
          continue;
        } else {
          idx[off] = (int32_t)x;
          const float w = pv[i] / qv[i];
          wc[off] = (h.mode == kDirect) ? w : ldexpf(w, h.scale);
          qc[off] = qv[i];
        }
        ++off;
      } else {
        rb[x] = 0.0f;
      }
    }
    running += total;
    __syncthreads();  // s_scan is reused by the next tile
  }
  if (!all_zero_weight) {
    const int npad = (int)round_up(h.n, K == 2 ? kBlockPolesPrep : 8);
    for (int j = h.n + tid; j < npad; j += kPrepThreads) {
      idx[j] = -1;
      wc[j] = 0.0f;
      qc[j] = 0.0f;
    }
  }
}

// ------------------------------------------------------------------ pole stream
// Per row, the poles (w', q) of the compacted support become a stream of
// 2 floats per pole: for the rational modes chunk c of C poles holds
// [e_1 .. e_C, n_{C-1} .. n_0] with D(a) = a^C + e_1 a^(C-1) + ... + e_C and
// N(a) = n_{C-1} a^(C-1) + ... + n_0 (coefficients formed in fp64); for the
// direct mode the stream is the interleaved pairs (w', q).  One thread per
// group of 8 poles.
// Coefficients of one chunk of C poles, fp64: D(a) = prod_c (a + w_c) and
// N(a) = sum_c q_c prod_{c' != c} (a + w_c'), written highest power first
// (the leading 1 of D is implicit).  N uses prefix and suffix products of the
// linear factors, so every coefficient is a sum of non-negative terms.
template <int C>
__device__ __forceinline__ void chunk_coefficients(const float* __restrict__ w, const float* __restrict__ q,
                                                   float* __restrict__ o) {
  // pre[c]: prod_{c' < c} (a + w_c'), degree c; coefficient k multiplies a^(c - k)
  double pre[C][C];
  double suf[C + 1][C + 1];
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int k = 0; k < C; ++k) pre[c][k] = (c == 0 && k == 0) ? 1.0 : 0.0;
#pragma unroll
  for (int c = 1; c < C; ++c) {
    const double wc = w[c - 1];
#pragma unroll
    for (int k = 0; k < C; ++k) pre[c][k] = (k <= c - 1 ? pre[c - 1][k] : 0.0) + (k >= 1 ? pre[c - 1][k - 1] * wc : 0.0);
  }
  // suf[c]: prod_{c' >= c} (a + w_c'), degree C - c
#pragma unroll
  for (int k = 0; k <= C; ++k) suf[C][k] = (k == 0) ? 1.0 : 0.0;
#pragma unroll
  for (int c = C - 1; c >= 0; --c) {
    const double wc = w[c];
#pragma unroll
    for (int k = 0; k <= C; ++k)
      suf[c][k] = (k <= C - c - 1 ? suf[c + 1][k] : 0.0) + (k >= 1 ? suf[c + 1][k - 1] * wc : 0.0);
  }
  // D = suf[0] (degree C, leading 1)
#pragma unroll
  for (int k = 1; k <= C; ++k) o[k - 1] = (float)suf[0][k];
  // N = sum_c q_c pre[c] * suf[c + 1]   (degree C - 1)
  double nn[C];
#pragma unroll
  for (int k = 0; k < C; ++k) nn[k] = 0.0;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const double qc = q[c];
    // pre[c] has degree c, suf[c+1] degree C-1-c; product coefficient k (k = 0..C-1)
#pragma unroll
    for (int i = 0; i < C; ++i) {
      if (i > c) continue;
#pragma unroll
      for (int j = 0; j < C; ++j) {
        if (j > C - 1 - c) continue;
        nn[i + j] += qc * pre[c][i] * suf[c + 1][j];
      }
    }
  }
#pragma unroll
  for (int k = 0; k < C; ++k) o[C + k] = (float)nn[k];
}

__global__ __launch_bounds__(256) void pole_stream_kernel(Workspace ws, int K) {
  const int64_t b = blockIdx.y;
  const RowHdr h = ws.hdr[b];
  if (h.mode == kSkip) return;
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const float* wc = ws.wc + b * ws.Sp;
  const float* qc = ws.qc + b * ws.Sp;
  float* out = ws.stream + b * ws.ld;
  if (K == 2 && h.mode != kDirect) return;  // packed by pole_pack_mfma_kernel
  // groups of 8 poles: interleaved (w', q) pairs, or K = 3 chunks stored contiguously
  const int npad = (int)round_up(h.n, 8);
  if (8 * u >= npad) return;
  const float* w8 = wc + 8 * u;
  const float* q8 = qc + 8 * u;
  float* o8 = out + 16 * u;
  if (h.mode == kDirect) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      o8[2 * i] = w8[i];
      o8[2 * i + 1] = q8[i];
    }
  } else if (h.mode == kRat8) {
    chunk_coefficients<8>(w8, q8, o8);
  } else {
    chunk_coefficients<4>(w8, q8, o8);
    chunk_coefficients<4>(w8 + 4, q8 + 4, o8 + 8);
  }
}

// ------------------------------------------------------------------ chunk evaluation
// Adds the chunks of an LDS tile to R running fp32 sums.
template <int R>
__device__ __forceinline__ void sweep_rat4(const float4* __restrict__ t, int nchunks, const float (&a)[R],
                                           float (&s)[R]) {
  for (int c = 0; c < nchunks; ++c) {
    const float4 e = t[2 * c], n = t[2 * c + 1];
#pragma unroll
    for (int i = 0; i < R; ++i) {
      float D = a[i] + e.x;
      D = fmaf(D, a[i], e.y);
      D = fmaf(D, a[i], e.z);
      D = fmaf(D, a[i], e.w);
      float N = fmaf(n.x, a[i], n.y);
      N = fmaf(N, a[i], n.z);
      N = fmaf(N, a[i], n.w);
      s[i] = fmaf(N, __builtin_amdgcn_rcpf(D), s[i]);
    }
  }
}

template <int R>
__device__ __forceinline__ void sweep_rat8(const float4* __restrict__ t, int nchunks, const float (&a)[R],
                                           float (&s)[R]) {
  for (int c = 0; c < nchunks; ++c) {
    const float4 e0 = t[4 * c], e1 = t[4 * c + 1], n0 = t[4 * c + 2], n1 = t[4 * c + 3];
#pragma unroll
    for (int i = 0; i < R; ++i) {
      float D = a[i] + e0.x;
      D = fmaf(D, a[i], e0.y);
      D = fmaf(D, a[i], e0.z);
      D = fmaf(D, a[i], e0.w);
      D = fmaf(D, a[i], e1.x);
      D = fmaf(D, a[i], e1.y);
      D = fmaf(D, a[i], e1.z);
      D = fmaf(D, a[i], e1.w);
      float N = fmaf(n0.x, a[i], n0.y);
      N = fmaf(N, a[i], n0.z);
      N = fmaf(N, a[i], n0.w);
      N = fmaf(N, a[i], n1.x);
      N = fmaf(N, a[i], n1.y);
      N = fmaf(N, a[i], n1.z);
      N = fmaf(N, a[i], n1.w);
      s[i] = fmaf(N, __builtin_amdgcn_rcpf(D), s[i]);
    }
  }
}

// Direct pairs (w', q), two per float4.
template <int R>
__device__ __forceinline__ void sweep_direct(const float4* __restrict__ t, int npairs2, const float (&a)[R],
                                             float (&s)[R]) {
  for (int c = 0; c < npairs2; ++c) {
    const float4 v = t[c];
#pragma unroll
    for (int i = 0; i < R; ++i) {
      s[i] = fmaf(v.y, __builtin_amdgcn_rcpf(a[i] + v.x), s[i]);
      s[i] = fmaf(v.w, __builtin_amdgcn_rcpf(a[i] + v.z), s[i]);
    }
  }
}

__device__ __forceinline__ void write_r(int64_t b, int64_t V, int K, const RowHdr& h, int32_t y, double S,
                                        const float* __restrict__ p, const float* __restrict__ q,
                                        float* __restrict__ r) {
  const float pv = p[b * V + y];
  double v;
  if (pv == 0.0f) {
    v = (double)q[b * V + y] * (K == 2 ? h.q0 : h.q0 * h.q0);
  } else {
    v = (double)K * (double)pv * ldexp(S, h.scale);
    // K = 2: the zero-weight tokens are not poles; each adds p(y) q(x) / w(y) = q(y) q(x)
    if (K == 2) v += 2.0 * (double)q[b * V + y] * h.q0;
  }
  r[b * V + y] = (float)v;
}

// Result of a K = 2 sweep for query j of row b: with one pole split, r is
// written directly (identical drafts) or the unscaled sum is stored by token
// into `dense` (two draft distributions); otherwise the split's partial sum.
__device__ __forceinline__ void store_sum(int64_t b, int64_t V, const RowHdr& h, int j, int split, double S,
                                          const Workspace& wq, double* __restrict__ dense,
                                          const float* __restrict__ p, const float* __restrict__ q,
                                          float* __restrict__ r) {
  if (wq.P > 1) {
    wq.part[(b * wq.P + split) * wq.Sp + j] = S;
  } else if (dense) {
    dense[b * V + wq.idx[b * wq.Sp + j]] = S;
  } else {
    write_r(b, V, 2, h, wq.idx[b * wq.Sp + j], S, p, q, r);
  }
}

// ------------------------------------------------------------------ K = 2 sweep, direct rows
// Rows whose weight range is too wide for the rational form: one reciprocal
// per (query, pole).  grid (query blocks of 256 * R, pole splits P, rows B);
// each lane holds R queries; the (w', q) pairs of the split are staged through
// LDS tile by tile (double buffered through registers) and read as broadcasts.
template <int R>
__global__ __launch_bounds__(kSweepThreads) void sweep_k2_direct_kernel(const float* __restrict__ p,
                                                                  const float* __restrict__ q, int64_t V,
                                                                  float* __restrict__ r, Workspace wq, Workspace wp,
                                                                  double* __restrict__ dense) {
  const int64_t b = blockIdx.z;
  const int split = blockIdx.y;
  const RowHdr h = wq.hdr[b];
  if (h.mode != kDirect) return;
  const int n = h.n;
  const int npole = wp.hdr[b].n;
  const int y0 = blockIdx.x * (kSweepThreads * R);
  if (y0 >= n) return;
  const int tid = threadIdx.x;
  // the pairs are split in groups of 8 poles (16 floats)
  const int ngroups = (int)(round_up(npole, 8) / 8);
  const int g_lo = (int)((int64_t)ngroups * split / wq.P);
  const int g_hi = (int)((int64_t)ngroups * (split + 1) / wq.P);
  const float* stream = wp.stream + b * wp.ld;
  const int64_t f_lo = 16 * (int64_t)g_lo, f_hi = 16 * (int64_t)g_hi;  // float range of the split

  float a[R];
  double acc[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int j = y0 + i * kSweepThreads + tid;
    a[i] = (j < n) ? wq.wc[b * wq.Sp + j] : 1.0f;
    acc[i] = 0.0;
  }
  __shared__ float4 tile[kTileFloats / 4];
  const float4* src = reinterpret_cast<const float4*>(stream);
  float4 reg0 = make_float4(0.f, 0.f, 0.f, 0.f), reg1 = reg0;
  auto fetch = [&](int64_t f0) {
    const int64_t i0 = f0 / 4 + tid, i1 = i0 + kSweepThreads;
    reg0 = (4 * i0 < f_hi) ? src[i0] : make_float4(0.f, 0.f, 0.f, 0.f);
    reg1 = (4 * i1 < f_hi) ? src[i1] : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  if (f_lo < f_hi) fetch(f_lo);
  for (int64_t f0 = f_lo; f0 < f_hi; f0 += kTileFloats) {
    __syncthreads();  // previous tile fully consumed
    tile[tid] = reg0;
    tile[tid + kSweepThreads] = reg1;
    __syncthreads();
    if (f0 + kTileFloats < f_hi) fetch(f0 + kTileFloats);
    const int nf = (int)min((int64_t)kTileFloats, f_hi - f0);
    // fold every 128 pairs to keep fp32 partial sums short
    for (int g = 0; g < nf / 4; g += 64) {
      float s2[R];
#pragma unroll
      for (int i = 0; i < R; ++i) s2[i] = 0.0f;
      sweep_direct<R>(tile + g, min(64, nf / 4 - g), a, s2);
#pragma unroll
      for (int i = 0; i < R; ++i) acc[i] += (double)s2[i];
    }
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int j = y0 + i * kSweepThreads + tid;
    if (j >= n) continue;
    store_sum(b, V, h, j, split, acc[i], wq, dense, p, q, r);
  }
}

// ------------------------------------------------------------------ K = 2 sweep, matrix cores
// For a tile of 16 queries (rows i) and 16 chunks (columns j) the chunk
// polynomials are a small dense contraction over the power index m:
//   D[i][j] = a_i^C + sum_{m<C} a_i^m d_m(j),   N[i][j] = sum_{m<C} a_i^m n_m(j)
// (d_m = e_{C-m}).  It runs on the bf16 matrix cores at fp32 accuracy: every
// fp32 operand x is split exactly into three bf16 parts x = x_h + x_m + x_l,
// and each product keeps the six cross terms above 2^-24 relative size,
//   a b ~ a_h b_h + a_h b_m + a_m b_h + a_h b_l + a_m b_m + a_l b_h,
// laid out along the contraction index k = 6 m + slot.  Products of bf16
// values are exact in the fp32 accumulator; every term of D and N is
// non-negative up to the small signed split corrections, so there is no
// cancellation.  The monic a^C is the accumulator input.  The VALU then adds
// N/D per output (one reciprocal per query and chunk).
//   C = 8: k in [0, 48): v_mfma_f32_16x16x32_bf16 for k < 32, then
//          v_mfma_f32_16x16x16_bf16 for k in [32, 48); 128-pole blocks, 3 KB.
//   C = 4: k in [0, 24), padded to 32: one 16x16x32 MFMA; 64-pole blocks, 2 KB.
// Block layout: planes of 64 lanes x 16 bytes (conflict-free ds_read_b128);
// lane L = 16 g + j holds the operand column j for k in its lane group g.
//   C = 8: plane 0 d (k = 8 g + e), plane 1 n (k = 8 g + e), plane 2 d then n (k = 32 + 4 g + e)
//   C = 4: plane 0 d (k = 8 g + e), plane 1 n (k = 8 g + e)
// Each wave holds MT M-tiles; workgroups are remapped so that each of the 8
// XCDs takes a contiguous range (the query blocks of a row share one L2).
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int kBlockPoles = 128;        // poles per padded K = 2 block (C = 8 block)
constexpr int kMfmaTileF4 = 1536;       // LDS tile: 24 KB of operand blocks
constexpr int kMfmaMT = MDSS_MFMA_MT;   // 16-query M-tiles per wave
constexpr int kMfmaNW = MDSS_MFMA_NW;   // waves per workgroup
constexpr int kMfmaThreads = 64 * kMfmaNW;
constexpr int kMfmaQueries = 16 * kMfmaMT * kMfmaNW;  // queries per workgroup

// exact split x = h + m + l into bf16 parts (each residual is exact in fp32)
__device__ __forceinline__ void split3(float x, float (&c)[3]) {
  const __bf16 h = (__bf16)x;
  const float r1 = x - (float)h;
  const __bf16 m = (__bf16)r1;
  const float r2 = r1 - (float)m;
  c[0] = (float)h;
  c[1] = (float)m;
  c[2] = (float)(__bf16)r2;
}
// product slots along k: (a part, b part) = (h,h) (h,m) (m,h) (h,l) (m,m) (l,h)
__device__ __forceinline__ int slot_a(int s) { return (s == 2 || s == 4) ? 1 : (s == 5 ? 2 : 0); }
__device__ __forceinline__ int slot_b(int s) { return (s == 1 || s == 4) ? 1 : (s == 3 ? 2 : 0); }
__device__ __forceinline__ float pick3(const float (&c)[3], int i) { return i == 0 ? c[0] : (i == 1 ? c[1] : c[2]); }

__device__ __forceinline__ float4 pack_bf16x8(const float (&v)[8]) {
  bf16x8 t;
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = (__bf16)v[e];
  return __builtin_bit_cast(float4, t);
}

// Packs the rational chunks of a K = 2 row into the bf16 operand blocks, one
// thread per chunk: the 8 bf16 values of one lane's float4 (its k range for
// column j) all come from the same chunk j, so a thread forms its chunk's
// coefficients (fp64, rounded to fp32), splits each once and writes its
// 12 (C = 8) or 8 (C = 4) float4s; threads j = 0..15 of a block write 16
// adjacent float4s per (plane, lane group).
template <int C>
__device__ __forceinline__ void pack_chunk(const float* __restrict__ w, const float* __restrict__ q,
                                           float4* __restrict__ blk, int j) {
  float o[16];
  chunk_coefficients<C>(w, q, o);  // o[k - 1] = e_k, o[C + k] = coefficient of a^(C - 1 - k) in N
  float dp[C][3], np[C][3];        // split parts of d_m = e_{C-m} and n_m
#pragma unroll
  for (int m = 0; m < C; ++m) {
    split3(o[C - 1 - m], dp[m]);
    split3(o[2 * C - 1 - m], np[m]);
  }
  constexpr int kPlanes = (C == 8) ? 3 : 2;
#pragma unroll
  for (int plane = 0; plane < kPlanes; ++plane)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        int k;
        bool is_n;
        if (plane < 2) {
          k = 8 * g + e;
          is_n = (plane == 1);
        } else {
          k = 32 + 4 * g + (e & 3);
          is_n = (e >= 4);
        }
        const int m = k / 6, sl = k % 6;
        v[e] = (m < C) ? (is_n ? np[m][slot_b(sl)] : dp[m][slot_b(sl)]) : 0.0f;
      }
      blk[plane * 64 + 16 * g + j] = pack_bf16x8(v);
    }
}

__global__ __launch_bounds__(256) void pole_pack_mfma_kernel(Workspace ws) {
  const int64_t b = blockIdx.y;
  const RowHdr h = ws.hdr[b];
  if (h.mode != kRat8 && h.mode != kRat4) return;
  const int C = h.mode;
  const int64_t nch = round_up(h.n, kBlockPoles) / C;
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= nch) return;
  const float* wc = ws.wc + b * ws.Sp;
  const float* qc = ws.qc + b * ws.Sp;
  float4* out = reinterpret_cast<float4*>(ws.stream + b * ws.ld);
  if (C == 8) {
    pack_chunk<8>(wc + 8 * c, qc + 8 * c, out + (c / 16) * 192, (int)(c % 16));
  } else {
    pack_chunk<4>(wc + 4 * c, qc + 4 * c, out + (c / 16) * 128, (int)(c % 16));
  }
}

// D and N of one operand block for the MT M-tiles (all MFMAs issued before any result is read).
template <int C, int MT>
__device__ __forceinline__ void mfma_block(const float4* __restrict__ blk, int lane, const bf16x8 (&AX)[MT],
                                           const bf16x4 (&AY)[MT], const f32x4 (&cinit)[MT], f32x4 (&D)[MT],
                                           f32x4 (&N)[MT]) {
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  const bf16x8 dx = __builtin_bit_cast(bf16x8, blk[lane]);
  const bf16x8 nx = __builtin_bit_cast(bf16x8, blk[64 + lane]);
  if (C == 8) {
    const float4 yy = blk[128 + lane];
    const bf16x4 dy = __builtin_bit_cast(bf16x4, make_float2(yy.x, yy.y));
    const bf16x4 ny = __builtin_bit_cast(bf16x4, make_float2(yy.z, yy.w));
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      D[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(AX[t], dx, cinit[t], 0, 0, 0);
      N[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(AX[t], nx, zero, 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      D[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(AY[t], dy, D[t], 0, 0, 0);
      N[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(AY[t], ny, N[t], 0, 0, 0);
    }
  } else {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      D[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(AX[t], dx, cinit[t], 0, 0, 0);
      N[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(AX[t], nx, zero, 0, 0, 0);
    }
  }
}

// acc += N / D for the outputs of one block
template <int MT>
__device__ __forceinline__ void mfma_consume(const f32x4 (&D)[MT], const f32x4 (&N)[MT], float (&acc)[MT][4]) {
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[t][r] = fmaf(N[t][r], __builtin_amdgcn_rcpf(D[t][r]), acc[t][r]);
}

template <int C, int MT>
__device__ __forceinline__ void mfma_sweep(const float4* __restrict__ src, int nblocks, int tid, int lane,
                                           const bf16x8 (&AX)[MT], const bf16x4 (&AY)[MT],
                                           const f32x4 (&cinit)[MT], double (&acc64)[MT][4],
                                           float4* __restrict__ tile) {
  constexpr int F = (C == 8) ? 192 : 128;           // float4 per block
  constexpr int kTileBlocks = kMfmaTileF4 / F;      // 8 or 12 blocks per LDS tile
  constexpr int kLoads = kMfmaTileF4 / kMfmaThreads;  // float4 per thread per tile
  const int64_t total_f4 = (int64_t)nblocks * F;
  float4 reg[kLoads];
  auto fetch = [&](int blk0) {
#pragma unroll
    for (int k = 0; k < kLoads; ++k) {
      const int64_t i = (int64_t)blk0 * F + k * kMfmaThreads + tid;
      reg[k] = (i < total_f4) ? src[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  if (nblocks > 0) fetch(0);
  for (int blk0 = 0; blk0 < nblocks; blk0 += kTileBlocks) {
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kLoads; ++k) tile[k * kMfmaThreads + tid] = reg[k];
    __syncthreads();
    if (blk0 + kTileBlocks < nblocks) fetch(blk0 + kTileBlocks);
    const int nb = min(kTileBlocks, nblocks - blk0);
    float acc[MT][4];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[t][r] = 0.0f;
    // software pipeline: the MFMAs of block bi + 1 are issued before the VALU work of block bi
    f32x4 D0[MT], N0[MT], D1[MT], N1[MT];
    mfma_block<C, MT>(tile, lane, AX, AY, cinit, D0, N0);
    int bi = 1;
    for (; bi + 1 < nb; bi += 2) {
      mfma_block<C, MT>(tile + bi * F, lane, AX, AY, cinit, D1, N1);
      mfma_consume<MT>(D0, N0, acc);
      mfma_block<C, MT>(tile + (bi + 1) * F, lane, AX, AY, cinit, D0, N0);
      mfma_consume<MT>(D1, N1, acc);
    }
    if (bi < nb) {
      mfma_block<C, MT>(tile + bi * F, lane, AX, AY, cinit, D1, N1);
      mfma_consume<MT>(D0, N0, acc);
      mfma_consume<MT>(D1, N1, acc);
    } else {
      mfma_consume<MT>(D0, N0, acc);
    }
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc64[t][r] += (double)acc[t][r];
  }
}

__global__ __launch_bounds__(kMfmaThreads) void sweep_k2_mfma_kernel(const float* __restrict__ p,
                                                                      const float* __restrict__ q, int64_t V,
                                                                      float* __restrict__ r, Workspace wq, Workspace wp,
                                                                      double* __restrict__ dense, int nqb,
                                                                      int64_t total) {
  constexpr int MT = kMfmaMT;
  // XCD-aware mapping: hardware block h runs on XCD h % 8; give each XCD a contiguous logical range
  const int64_t hw = blockIdx.x;
  const int64_t per = total / 8, rem = total % 8, x = hw % 8;
  const int64_t logical = x * per + (x < rem ? x : rem) + hw / 8;
  const int qb = (int)(logical % nqb);
  const int64_t rest = logical / nqb;
  const int split = (int)(rest % wq.P);
  const int64_t b = rest / wq.P;
  const RowHdr h = wq.hdr[b];
  if (h.mode != kRat8 && h.mode != kRat4) return;
  const int n = h.n;
  const int npole = wp.hdr[b].n;
  const int q0 = qb * kMfmaQueries;
  if (q0 >= n) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, col = lane & 15;
  const int C = h.mode;
  const float* wc = wq.wc + b * wq.Sp;

  // A[i][k] = part slot_a(k % 6) of a_i^(k / 6) (row i = col); accumulator input a^C for rows 4 g + r
  bf16x8 AX[MT];
  bf16x4 AY[MT];
  f32x4 cinit[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int base = q0 + 16 * (MT * wave + t);
    const float a = (base + col < n) ? wc[base + col] : 1.0f;
    float pw[8];
    pw[0] = 1.0f;
#pragma unroll
    for (int m = 1; m < 8; ++m) pw[m] = pw[m - 1] * a;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 8 * g + e, m = k / 6, sl = k % 6;
      float parts[3];
      float pm = pw[0];
#pragma unroll
      for (int mm = 1; mm < 8; ++mm) pm = (m == mm) ? pw[mm] : pm;
      split3(pm, parts);
      AX[t][e] = (__bf16)((m < C) ? pick3(parts, slot_a(sl)) : 0.0f);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = 32 + 4 * g + e, m = k / 6, sl = k % 6;
      float parts[3];
      float pm = pw[0];
#pragma unroll
      for (int mm = 1; mm < 8; ++mm) pm = (m == mm) ? pw[mm] : pm;
      split3(pm, parts);
      AY[t][e] = (__bf16)((m < C) ? pick3(parts, slot_a(sl)) : 0.0f);
    }
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int qi = base + 4 * g + rr;
      const float ar = (qi < n) ? wc[qi] : 1.0f;
      const float ar2 = ar * ar, ar4 = ar2 * ar2;
      cinit[t][rr] = (C == 8) ? ar4 * ar4 : ar4;
    }
  }
  const int poles_per_block = (C == 8) ? 128 : 64;
  const int F = (C == 8) ? 192 : 128;
  const int nblocks = (int)(round_up(npole, kBlockPoles) / poles_per_block);
  const int b_lo = (int)((int64_t)nblocks * split / wq.P);
  const int b_hi = (int)((int64_t)nblocks * (split + 1) / wq.P);
  const float4* src = reinterpret_cast<const float4*>(wp.stream + b * wp.ld) + (int64_t)b_lo * F;
  __shared__ float4 tile[kMfmaTileF4];
  double acc64[MT][4];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) acc64[t][rr] = 0.0;
  if (C == 8) {
    mfma_sweep<8, MT>(src, b_hi - b_lo, tid, lane, AX, AY, cinit, acc64, tile);
  } else {
    mfma_sweep<4, MT>(src, b_hi - b_lo, tid, lane, AX, AY, cinit, acc64, tile);
  }
  // each query row is spread over the 16 lanes of its group (one chunk column each)
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      double v = acc64[t][rr];
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off, 64);
      acc64[t][rr] = v;
    }
  if (col == 0) {
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int qi = q0 + 16 * (MT * wave + t) + 4 * g + rr;
        if (qi >= n) continue;
        store_sum(b, V, h, qi, split, acc64[t][rr], wq, dense, p, q, r);
      }
  }
}

// ------------------------------------------------------------------ K = 3 sweep
// r(y) = 3 p(y) sum_{x2} q(x2) [ q(x2)/(a2 + w(x2)) + 2 sum_{x3 > x2} q(x3)/(a2 + w(x3)) ],
// a2 = w(y) + w(x2) (unordered {x2, x3} pairs, diagonal once).  The whole
// compacted row (<= s_max poles) and its pole stream live in LDS; grid
// (query blocks, x2 splits P, rows B) with x2 ranges of equal triangular work.
template <int R>
__global__ __launch_bounds__(kSweepThreads) void sweep_k3_kernel(Workspace ws) {
  extern __shared__ float4 lds[];
  const int64_t b = blockIdx.z;
  const int split = blockIdx.y;
  const RowHdr h = ws.hdr[b];
  if (h.mode == kSkip) return;
  const int n = h.n;
  const int y0 = blockIdx.x * (kSweepThreads * R);
  if (y0 >= n) return;
  const int tid = threadIdx.x;
  const int C = mode_chunk(h.mode);
  const int npad = (int)round_up(n, 8);
  const int nchunks = npad / C;  // includes the zero padding poles, which add nothing

  // LDS: [w' (npad)] [q (npad)] [stream (2 npad)]
  float* s_w = reinterpret_cast<float*>(lds);
  float* s_q = s_w + npad;
  float4* s_stream = reinterpret_cast<float4*>(s_q + npad);
  const float* gw = ws.wc + b * ws.Sp;
  const float* gq = ws.qc + b * ws.Sp;
  const float4* gs = reinterpret_cast<const float4*>(ws.stream + b * ws.ld);
  for (int j = tid; j < npad; j += kSweepThreads) {
    s_w[j] = gw[j];
    s_q[j] = gq[j];
  }
  for (int j = tid; j < npad / 2; j += kSweepThreads) s_stream[j] = gs[j];
  __syncthreads();

  // x2 range with equal shares of sum_{x2} (n - x2) work
  const double T = 0.5 * (double)n * (double)(n + 1);
  auto bound = [&](int k) -> int {
    if (k <= 0) return 0;
    if (k >= ws.P) return n;
    const double np = (double)n + 0.5;
    const double m = np - sqrt(np * np - 2.0 * T * (double)k / (double)ws.P);
    return min(n, max(0, (int)llround(m)));
  };
  const int x2_lo = bound(split), x2_hi = bound(split + 1);

  float a[R];
  double acc[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int j = y0 + i * kSweepThreads + tid;
    a[i] = (j < n) ? s_w[j] : 1.0f;
    acc[i] = 0.0;
  }
  for (int x2 = x2_lo; x2 < x2_hi; ++x2) {
    const float w2 = s_w[x2], q2 = s_q[x2];
    float a2[R], off[R], dg[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
      a2[i] = a[i] + w2;
      off[i] = 0.0f;
      dg[i] = q2 * __builtin_amdgcn_rcpf(a2[i] + w2);
    }
    if (h.mode == kDirect) {
      for (int x3 = x2 + 1; x3 < n; ++x3) {
        const float w3 = s_w[x3], q3 = s_q[x3];
#pragma unroll
        for (int i = 0; i < R; ++i) off[i] = fmaf(q3, __builtin_amdgcn_rcpf(a2[i] + w3), off[i]);
      }
    } else {
      const int c2 = x2 / C;
      const int head_end = min((c2 + 1) * C, n);
      for (int x3 = x2 + 1; x3 < head_end; ++x3) {
        const float w3 = s_w[x3], q3 = s_q[x3];
#pragma unroll
        for (int i = 0; i < R; ++i) off[i] = fmaf(q3, __builtin_amdgcn_rcpf(a2[i] + w3), off[i]);
      }
      const int cstart = c2 + 1;
      if (cstart < nchunks) {
        if (C == 8) {
          sweep_rat8<R>(s_stream + 4 * cstart, nchunks - cstart, a2, off);
        } else {
          sweep_rat4<R>(s_stream + 2 * cstart, nchunks - cstart, a2, off);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < R; ++i) acc[i] += (double)q2 * ((double)dg[i] + 2.0 * (double)off[i]);
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int j = y0 + i * kSweepThreads + tid;
    if (j < n) ws.part[(b * ws.P + split) * ws.Sp + j] = acc[i];
  }
}

// Sum the P partial sums of each support entry in split order and write r.
__global__ __launch_bounds__(256) void finalize_kernel(const float* __restrict__ p, const float* __restrict__ q,
                                                        int64_t V, int K, float* __restrict__ r, Workspace ws) {
  const int64_t b = blockIdx.y;
  const RowHdr h = ws.hdr[b];
  if (h.mode == kSkip) return;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= h.n) return;
  double S = 0.0;
  for (int s = 0; s < ws.P; ++s) S += ws.part[(b * ws.P + s) * ws.Sp + j];
  write_r(b, V, K, h, ws.idx[b * ws.Sp + j], S, p, q, r);
}


// ------------------------------------------------------------------ two draft distributions (K = 2)
// Drafts X1 ~ q1, X2 ~ q2 with the classical weights w_i = p / q_i (Remark 1;
// the non-identical K = 2 appendix).  Splitting the drafted pairs by which
// index holds y gives
//   r(y) = p(y) [ S_2(w_1(y)) + S_1(w_2(y)) ],  S_i(a) = sum_{x in supp q_i} q_i(x) / (a + w_i(x)),
// the first term only when q1(y) > 0 and the second only when q2(y) > 0;
// a zero-target token gets (q1(y) Q2_0 + q2(y) Q1_0) / 2, Qi_0 the q_i-mass of
// the zero-weight tokens of draft i (both weights zero: uniform index).
// Each S_i is one sweep of the K = 2 kernels with the queries of one draft
// and the poles of the other, sharing one scale over both drafts' weights.
__global__ __launch_bounds__(kPrepThreads) void prep_pair_kernel(const float* __restrict__ p,
                                                                  const float* __restrict__ q1,
                                                                  const float* __restrict__ q2, int64_t V,
                                                                  float* __restrict__ r,
                                                                  int32_t* __restrict__ row_status, Workspace w1,
                                                                  Workspace w2) {
  const int64_t b = blockIdx.x;
  const float* pb = p + b * V;
  const float* ab = q1 + b * V;
  const float* cb = q2 + b * V;
  float* rb = r + b * V;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int kWaves = kPrepThreads / 64;
  __shared__ double s_z1[kWaves], s_z2[kWaves];
  __shared__ int s_n1[kWaves], s_n2[kWaves], s_bad[kWaves];
  __shared__ float s_wmin[kWaves], s_wmax[kWaves];
  __shared__ int s_scan1[kWaves], s_scan2[kWaves];
  __shared__ RowHdr s_h1, s_h2;

  int bad = 0, n1 = 0, n2 = 0;
  double z1 = 0.0, z2 = 0.0;
  float wmin = INFINITY, wmax = 0.0f;
  for (int64_t x = tid; x < V; x += kPrepThreads) {
    const float pv = pb[x], av = ab[x], cv = cb[x];
    bad |= (int)(bad_prob(pv) || bad_prob(av) || bad_prob(cv));
    if (av > 0.0f) {
      n1 += pv > 0.0f;
      if (pv == 0.0f) {
        z1 += (double)av;
      } else {
        const float w = pv / av;
        wmin = fminf(wmin, w);
        wmax = fmaxf(wmax, w);
      }
    }
    if (cv > 0.0f) {
      n2 += pv > 0.0f;
      if (pv == 0.0f) {
        z2 += (double)cv;
      } else {
        const float w = pv / cv;
        wmin = fminf(wmin, w);
        wmax = fmaxf(wmax, w);
      }
    }
  }
  bad = wave_sum_int(bad);
  n1 = wave_sum_int(n1);
  n2 = wave_sum_int(n2);
  z1 = wave_sum(z1);
  z2 = wave_sum(z2);
  wmin = wave_min(wmin);
  wmax = wave_max(wmax);
  if (lane == 0) {
    s_bad[wid] = bad;
    s_n1[wid] = n1;
    s_n2[wid] = n2;
    s_z1[wid] = z1;
    s_z2[wid] = z2;
    s_wmin[wid] = wmin;
    s_wmax[wid] = wmax;
  }
  __syncthreads();
  if (tid == 0) {
    int tb = 0, t1 = 0, t2 = 0;
    double tz1 = 0.0, tz2 = 0.0;
    float mn = INFINITY, mx = 0.0f;
    for (int i = 0; i < kWaves; ++i) {
      tb |= s_bad[i];
      t1 += s_n1[i];
      t2 += s_n2[i];
      tz1 += s_z1[i];
      tz2 += s_z2[i];
      mn = fminf(mn, s_wmin[i]);
      mx = fmaxf(mx, s_wmax[i]);
    }
    RowHdr h;
    h.pad = 0.0;
    h.scale = 0;
    h.flags = tb ? kRowBadProb : 0;
    if (h.flags || !(mx > 0.0f)) {
      h.mode = kSkip;  // flagged, or no positive weight (every support token has p = 0)
    } else {
      int e_lo, e_hi;
      frexpf(mn, &e_lo);
      frexpf(mx, &e_hi);
      const int range = e_hi - e_lo;
      if (!isfinite(mx) || range > kRat4MaxRange) {
        h.mode = kDirect;
      } else {
        h.mode = range <= kRat8MaxRange ? kRat8 : kRat4;
        h.scale = -((e_lo + e_hi) >> 1);
      }
    }
    RowHdr h1 = h, h2 = h;
    h1.n = t1;
    h1.q0 = tz1;
    h2.n = t2;
    h2.q0 = tz2;
    s_h1 = h1;
    s_h2 = h2;
    w1.hdr[b] = h1;
    w2.hdr[b] = h2;
    if (row_status && h.flags) row_status[b] |= h.flags;
  }
  __syncthreads();
  const RowHdr h1 = s_h1, h2 = s_h2;
  if (h1.flags) {
    for (int64_t x = tid; x < V; x += kPrepThreads) rb[x] = NAN;
    return;
  }
  if (h1.mode == kSkip) return;  // r is formed by finalize_pair_kernel alone
  int run1 = 0, run2 = 0;
  for (int64_t base = 0; base < V; base += 4 * kPrepThreads) {
    const int64_t x0 = base + 4 * (int64_t)tid;
    float pv[4], av[4], cv[4];
    int c1 = 0, c2 = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t x = x0 + i;
      pv[i] = (x < V) ? pb[x] : 0.0f;
      av[i] = (x < V) ? ab[x] : 0.0f;
      cv[i] = (x < V) ? cb[x] : 0.0f;
      c1 += (av[i] > 0.0f) && (pv[i] > 0.0f);
      c2 += (cv[i] > 0.0f) && (pv[i] > 0.0f);
    }
    const int i1 = wave_inclusive_scan_int(c1, lane), i2 = wave_inclusive_scan_int(c2, lane);
    if (lane == 63) {
      s_scan1[wid] = i1;
      s_scan2[wid] = i2;
    }
    __syncthreads();
    int off1 = 0, off2 = 0, tot1 = 0, tot2 = 0;
    for (int i = 0; i < kWaves; ++i) {
      off1 += (i < wid) ? s_scan1[i] : 0;
      off2 += (i < wid) ? s_scan2[i] : 0;
      tot1 += s_scan1[i];
      tot2 += s_scan2[i];
    }
    int o1 = run1 + off1 + i1 - c1, o2 = run2 + off2 + i2 - c2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t x = x0 + i;
      if (x >= V) break;
      if (!(pv[i] > 0.0f)) continue;  // zero-weight tokens: closed form in finalize_pair_kernel
      if (av[i] > 0.0f) {
        const float w = pv[i] / av[i];
        w1.idx[b * w1.Sp + o1] = (int32_t)x;
        w1.wc[b * w1.Sp + o1] = (h1.mode == kDirect) ? w : ldexpf(w, h1.scale);
        w1.qc[b * w1.Sp + o1] = av[i];
        ++o1;
      }
      if (cv[i] > 0.0f) {
        const float w = pv[i] / cv[i];
        w2.idx[b * w2.Sp + o2] = (int32_t)x;
        w2.wc[b * w2.Sp + o2] = (h2.mode == kDirect) ? w : ldexpf(w, h2.scale);
        w2.qc[b * w2.Sp + o2] = cv[i];
        ++o2;
      }
    }
    run1 += tot1;
    run2 += tot2;
    __syncthreads();
  }
  const int np1 = (int)round_up(h1.n, kBlockPolesPrep), np2 = (int)round_up(h2.n, kBlockPolesPrep);
  for (int j = h1.n + tid; j < np1; j += kPrepThreads) {
    w1.idx[b * w1.Sp + j] = -1;
    w1.wc[b * w1.Sp + j] = 0.0f;
    w1.qc[b * w1.Sp + j] = 0.0f;
  }
  for (int j = h2.n + tid; j < np2; j += kPrepThreads) {
    w2.idx[b * w2.Sp + j] = -1;
    w2.wc[b * w2.Sp + j] = 0.0f;
    w2.qc[b * w2.Sp + j] = 0.0f;
  }
}

// Sum of the pole splits of each query, stored by token into `dense`.
__global__ __launch_bounds__(256) void dense_from_parts_kernel(int64_t V, Workspace wq, double* __restrict__ dense) {
  const int64_t b = blockIdx.y;
  const RowHdr h = wq.hdr[b];
  if (h.mode == kSkip) return;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= h.n) return;
  double S = 0.0;
  for (int s = 0; s < wq.P; ++s) S += wq.part[(b * wq.P + s) * wq.Sp + j];
  dense[b * V + wq.idx[b * wq.Sp + j]] = S;
}

__global__ __launch_bounds__(256) void finalize_pair_kernel(const float* __restrict__ p,
                                                             const float* __restrict__ q1,
                                                             const float* __restrict__ q2, int64_t V,
                                                             float* __restrict__ r, Workspace w1, Workspace w2,
                                                             const double* __restrict__ s_a,
                                                             const double* __restrict__ s_b) {
  const int64_t b = blockIdx.y;
  const RowHdr h1 = w1.hdr[b], h2 = w2.hdr[b];
  if (h1.flags) return;
  const int64_t y = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (y >= V) return;
  const int64_t i = b * V + y;
  const float pv = p[i], av = q1[i], cv = q2[i];
  double v = 0.0;
  // zero-weight poles of the other draft add p(y) q_j(x) / w_i(y) = q_i(y) q_j(x): q_i(y) Qj_0 in all
  if (av > 0.0f)
    v += (pv > 0.0f) ? (double)pv * ldexp(s_a[i], h1.scale) + (double)av * h2.q0 : 0.5 * (double)av * h2.q0;
  if (cv > 0.0f)
    v += (pv > 0.0f) ? (double)pv * ldexp(s_b[i], h1.scale) + (double)cv * h1.q0 : 0.5 * (double)cv * h1.q0;
  r[i] = (float)v;
}

constexpr int kK2R = 8;
constexpr int kK3R = 4;

}  // namespace

int choose_splits(int64_t B, int64_t V, int K, int s_max) {
  if (K == 2) {
    const int64_t yb = (V + kMfmaQueries - 1) / kMfmaQueries;
    const int64_t wgs = yb * B;
    int64_t P = (2048 + wgs - 1) / wgs;
    const int64_t max_p = std::max<int64_t>(1, V / 2048);  // keep >= 2048 poles per split
    P = std::min<int64_t>(P, std::min<int64_t>(16, max_p));
    return (int)std::max<int64_t>(P, 1);
  }
  const int64_t n = std::min<int64_t>(s_max, V);
  const int64_t yb = (n + kSweepThreads * kK3R - 1) / (kSweepThreads * kK3R);
  int64_t P = (4096 + yb * B - 1) / (yb * B);
  P = std::min<int64_t>(P, std::min<int64_t>(32, std::max<int64_t>(1, n / 16)));
  return (int)std::max<int64_t>(P, 1);
}

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// K = 2 rows hold packed bf16 operands: up to 32 bytes per pole (4-pole chunks)
static int64_t stream_ld(int K, int64_t Sp) { return K == 2 ? 8 * Sp : 2 * Sp; }

static int64_t padded_len(int64_t V, int K, int s_max) {
  return K == 2 ? round_up(V, kBlockPoles) : round_up(std::min<int64_t>(s_max, V), 8);
}

size_t workspace_bytes(int64_t B, int64_t V, int K, int s_max, int P) {
  const int64_t Sp = padded_len(V, K, s_max);
  size_t t = align256(sizeof(RowHdr) * B);
  t += 3 * align256(sizeof(float) * B * Sp);
  t += align256(sizeof(float) * stream_ld(K, Sp) * B);
  const bool need_part = (K == 3) || P > 1;
  if (need_part) t += align256(sizeof(double) * B * P * Sp);
  return t;
}

void carve_workspace(void* base, int64_t B, int64_t V, int K, int s_max, int P, Workspace* ws) {
  const int64_t Sp = padded_len(V, K, s_max);
  char* c = static_cast<char*>(base);
  ws->hdr = reinterpret_cast<RowHdr*>(c);
  c += align256(sizeof(RowHdr) * B);
  ws->idx = reinterpret_cast<int32_t*>(c);
  c += align256(sizeof(float) * B * Sp);
  ws->wc = reinterpret_cast<float*>(c);
  c += align256(sizeof(float) * B * Sp);
  ws->qc = reinterpret_cast<float*>(c);
  c += align256(sizeof(float) * B * Sp);
  ws->stream = reinterpret_cast<float*>(c);
  c += align256(sizeof(float) * stream_ld(K, Sp) * B);
  ws->part = ((K == 3) || P > 1) ? reinterpret_cast<double*>(c) : nullptr;
  ws->Sp = Sp;
  ws->ld = stream_ld(K, Sp);
  ws->P = P;
}

hipError_t launch_induced(const float* p, const float* q, int64_t B, int64_t V, int K, int s_max, float* r,
                          int32_t* row_status, const Workspace& ws, hipStream_t st) {
  hipLaunchKernelGGL(prep_kernel, dim3((unsigned)B), dim3(kPrepThreads), 0, st, p, q, V, K, s_max, r, row_status,
                     ws);
  const int64_t units = ws.Sp / 4;  // at most one thread per 4 poles
  hipLaunchKernelGGL(pole_stream_kernel, dim3((unsigned)((units + 255) / 256), (unsigned)B), dim3(256), 0, st, ws,
                     K);
  if (K == 2) {
    hipLaunchKernelGGL(pole_pack_mfma_kernel, dim3((unsigned)((ws.Sp / 4 + 255) / 256), (unsigned)B), dim3(256), 0,
                       st, ws);
    const int nqb = (int)((V + kMfmaQueries - 1) / kMfmaQueries);
    const int64_t total = (int64_t)nqb * ws.P * B;
    hipLaunchKernelGGL(sweep_k2_mfma_kernel, dim3((unsigned)total), dim3(kMfmaThreads), 0, st, p, q, V, r, ws, ws,
                       nullptr, nqb, total);
    const int64_t yb = (V + kSweepThreads * kK2R - 1) / (kSweepThreads * kK2R);
    hipLaunchKernelGGL(sweep_k2_direct_kernel<kK2R>, dim3((unsigned)yb, (unsigned)ws.P, (unsigned)B),
                       dim3(kSweepThreads), 0, st, p, q, V, r, ws, ws, nullptr);
  } else {
    const int64_t yb = (ws.Sp + kSweepThreads * kK3R - 1) / (kSweepThreads * kK3R);
    const size_t lds = sizeof(float) * 4 * ws.Sp;  // w', q, stream (2 per pole)
    hipLaunchKernelGGL(sweep_k3_kernel<kK3R>, dim3((unsigned)yb, (unsigned)ws.P, (unsigned)B), dim3(kSweepThreads),
                       lds, st, ws);
  }
  if (K == 3 || ws.P > 1) {
    hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)((ws.Sp + 255) / 256), (unsigned)B), dim3(256), 0, st, p, q,
                       V, K, r, ws);
  }
  return hipGetLastError();
}


size_t workspace_bytes_pair(int64_t B, int64_t V) {
  const int P = choose_splits(B, V, 2, 0);
  return 2 * workspace_bytes(B, V, 2, 0, P) + 2 * align256(sizeof(double) * B * V);
}

hipError_t launch_induced_pair(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, float* r,
                               int32_t* row_status, void* workspace, hipStream_t st) {
  const int P = choose_splits(B, V, 2, 0);
  const size_t one = workspace_bytes(B, V, 2, 0, P);
  Workspace w1, w2;
  char* base = static_cast<char*>(workspace);
  carve_workspace(base, B, V, 2, 0, P, &w1);
  carve_workspace(base + one, B, V, 2, 0, P, &w2);
  double* s_a = reinterpret_cast<double*>(base + 2 * one);
  double* s_b = reinterpret_cast<double*>(base + 2 * one + align256(sizeof(double) * B * V));
  hipLaunchKernelGGL(prep_pair_kernel, dim3((unsigned)B), dim3(kPrepThreads), 0, st, p, q1, q2, V, r, row_status, w1,
                     w2);
  const int64_t units = w1.Sp / 4;
  for (const Workspace* w : {&w1, &w2}) {
    hipLaunchKernelGGL(pole_stream_kernel, dim3((unsigned)((units + 255) / 256), (unsigned)B), dim3(256), 0, st, *w,
                       2);
    hipLaunchKernelGGL(pole_pack_mfma_kernel, dim3((unsigned)((units + 255) / 256), (unsigned)B), dim3(256), 0, st,
                       *w);
  }
  const int nqb = (int)((V + kMfmaQueries - 1) / kMfmaQueries);
  const int64_t total = (int64_t)nqb * P * B;
  const int64_t yb = (V + kSweepThreads * kK2R - 1) / (kSweepThreads * kK2R);
  // S_2 at the draft-1 weights, then S_1 at the draft-2 weights
  hipLaunchKernelGGL(sweep_k2_mfma_kernel, dim3((unsigned)total), dim3(kMfmaThreads), 0, st, p, q1, V, r, w1, w2, s_a,
                     nqb, total);
  hipLaunchKernelGGL(sweep_k2_direct_kernel<kK2R>, dim3((unsigned)yb, (unsigned)P, (unsigned)B), dim3(kSweepThreads),
                     0, st, p, q1, V, r, w1, w2, s_a);
  if (P > 1)
    hipLaunchKernelGGL(dense_from_parts_kernel, dim3((unsigned)((w1.Sp + 255) / 256), (unsigned)B), dim3(256), 0, st,
                       V, w1, s_a);
  hipLaunchKernelGGL(sweep_k2_mfma_kernel, dim3((unsigned)total), dim3(kMfmaThreads), 0, st, p, q2, V, r, w2, w1, s_b,
                     nqb, total);
  hipLaunchKernelGGL(sweep_k2_direct_kernel<kK2R>, dim3((unsigned)yb, (unsigned)P, (unsigned)B), dim3(kSweepThreads),
                     0, st, p, q2, V, r, w2, w1, s_b);
  if (P > 1)
    hipLaunchKernelGGL(dense_from_parts_kernel, dim3((unsigned)((w2.Sp + 255) / 256), (unsigned)B), dim3(256), 0, st,
                       V, w2, s_b);
  hipLaunchKernelGGL(finalize_pair_kernel, dim3((unsigned)((V + 255) / 256), (unsigned)B), dim3(256), 0, st, p, q1,
                     q2, V, r, w1, w2, s_a, s_b);
  return hipGetLastError();
}

// Successive pairwise reduction (Remark 4): r_1 = the K = 2 law of (q, q),
// r_j = the law of a pair drawn from (r_{j-1}, q), each stage read back in fp32.
hipError_t launch_induced_successive(const float* p, const float* q, int64_t B, int64_t V, int K, float* r_stages,
                                     int32_t* row_status, void* workspace, hipStream_t st) {
  const int P = choose_splits(B, V, 2, 0);
  Workspace ws;
  carve_workspace(workspace, B, V, 2, 0, P, &ws);
  hipError_t e = launch_induced(p, q, B, V, 2, 0, r_stages, row_status, ws, st);
  const int64_t plane = B * V;
  for (int j = 1; j < K - 1 && e == hipSuccess; ++j)
    e = launch_induced_pair(p, r_stages + (j - 1) * plane, q, B, V, r_stages + j * plane, row_status, workspace, st);
  return e;
}

}  // namespace mdss
