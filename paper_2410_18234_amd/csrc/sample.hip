// Selection of the intermediate token (Definition 1, index form with the
// classical weights) and single-draft speculative sampling of that token
// against the target (Algorithm 1), gfx950.
//
// Notation: p = target, q = draft, r = induced distribution of the selected
// token (the proposal of Algorithm 1).  Decisions are taken in fp64 with the
// uniforms as 24-bit dyadics, so the accept test u * r(Y) < p(Y) is exact.
#include "common.h"
#include "draw.h"

#include <algorithm>

#include <math.h>

namespace mdss {

namespace {

// ------------------------------------------------------------------ selection
// One thread per position.  q2 == nullptr: every draft from q; else K = 2 and
// draft i from q_{i+1} (two drafts from different distributions).
__global__ __launch_bounds__(256) void select_kernel(const float* __restrict__ p, const float* __restrict__ q,
                                                      const float* __restrict__ q2,
                                                      const int32_t* __restrict__ drafts,
                                                      const float* __restrict__ u, uint64_t seed, uint64_t offset,
                                                      int64_t B, int64_t V, int K, int32_t* __restrict__ sel_index,
                                                      int32_t* __restrict__ sel_token,
                                                      int32_t* __restrict__ row_status) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int st = 0;
  double w[kMaxK];
  int32_t x[kMaxK];
  for (int i = 0; i < K; ++i) {
    x[i] = drafts[b * K + i];
    const bool in = x[i] >= 0 && (int64_t)x[i] < V;
    const float* qi = (q2 != nullptr && i == 1) ? q2 : q;
    w[i] = draft_weight(in, in ? p[b * V + x[i]] : 0.0f, in ? qi[b * V + x[i]] : 0.0f, st);
  }
  if (st) {
    sel_index[b] = -1;
    sel_token[b] = -1;
    if (row_status) row_status[b] |= st;
    return;
  }
  float uu[3];
  position_uniforms(u, seed, offset, b, uu);
  const int istar = select_index(w, K, (double)uu[0]);
  sel_index[b] = istar;
  sel_token[b] = x[istar];
}


// Successive pairwise selection (Remark 4).  Stage 1 chooses between X1 and
// X2 (both from q, weights p/q); stage j >= 2 between the token Y kept so far
// (law r_{j-1}, weight p(Y)/r_{j-1}(Y)) and X_{j+1} (weight p/q).  Y is kept
// iff u_j (w_Y + w_X) < w_Y (fp64), or floor(2 u_j) = 0 when both weights are
// zero.  u_j = u_sel[b][j-1], else word 0 of Philox(seed, (offset + b, j)).
__global__ __launch_bounds__(256) void select_successive_kernel(
    const float* __restrict__ p, const float* __restrict__ q, const float* __restrict__ r_stages,
    const int32_t* __restrict__ drafts, const float* __restrict__ u_sel, uint64_t seed, uint64_t offset, int64_t B,
    int64_t V, int K, int32_t* __restrict__ sel_index, int32_t* __restrict__ sel_token,
    int32_t* __restrict__ row_status) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int st = 0;
  for (int i = 0; i < K; ++i) {
    const int32_t x = drafts[b * K + i];
    if (x < 0 || (int64_t)x >= V) {
      st |= kRowBadDraft;
      continue;
    }
    const float pv = p[b * V + x], qv = q[b * V + x];
    if (bad_prob(pv) || bad_prob(qv))
      st |= kRowBadProb;
    else if (!(qv > 0.0f))
      st |= kRowBadDraft;
  }
  int32_t y = -1;
  int idx = 0;
  if (!st) {
    y = drafts[b * K];
    for (int j = 1; j < K; ++j) {
      const int32_t x = drafts[b * K + j];
      const float ly = j == 1 ? q[b * V + y] : r_stages[(int64_t)(j - 2) * B * V + b * V + y];
      if (!(ly > 0.0f)) {
        st = kRowBadDraft;
        break;
      }
      const double wa = (double)p[b * V + y] / (double)ly;
      const double wb = (double)p[b * V + x] / (double)q[b * V + x];
      float u;
      if (u_sel) {
        u = u_sel[b * (K - 1) + (j - 1)];
      } else {
        const uint64_t pos = offset + (uint64_t)b;
        uint32_t c[4] = {(uint32_t)pos, (uint32_t)(pos >> 32), (uint32_t)j, 0u};
        philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
        u = (float)(c[0] >> 8) * 5.9604644775390625e-8f;  // 2^-24
      }
      const double W = wa + wb;
      const bool keep = W > 0.0 ? (double)u * W < wa : floor(2.0 * (double)u) == 0.0;
      if (!keep) {
        y = x;
        idx = j;
      }
    }
  }
  if (st) {
    sel_index[b] = -1;
    sel_token[b] = -1;
    if (row_status) row_status[b] |= st;
    return;
  }
  sel_index[b] = idx;
  sel_token[b] = y;
}


// ------------------------------------------------------------------ accept / resample
// Two forms, the same arithmetic (Algorithm 1 with proposal r; res = max(0, p - r)
// and its running sums in fp64).
// Row form (neither the residual nor its mass is asked for: only rejected
// positions read their rows): one workgroup of 8 waves per position.  The
// selection (fused form) and the accept test come first; a rejected position
// streams its row in 1024-token super-tiles (wave w takes super-tiles w, w + 8,
// w + 16, w + 24 in one pass, then the next 32), keeps each super-tile's
// residual sum in LDS and its last pass's p and r in registers; every wave then
// scans the sums, and the wave holding the crossing super-tile finds the token
// in it (a re-read only for rows longer than 32768 tokens whose crossing lies in
// an earlier pass).
// Segment form (the residual or its mass asked for: every position streams its
// row), two launches:
// (A) one workgroup per (position, segment of 4096 tokens): res = max(0, p - r)
//     over the segment in fp64 (stored as fp32 if asked for) and one fp64 sum per
//     256-token sub-tile (NaN when the sub-tile holds a bad probability);
// (B) one wave per position: the selection (fused form) and the accept test,
//     with the sub-tile sums read at the same time; Z from the sums in order,
//     the first sub-tile whose running sum exceeds u_res * Z, and the token
//     inside it from its 256 entries.
// A position's row is so spread over all of its segments' workgroups.
constexpr int kAccRowThreads = 512;
constexpr int kAccRowWaves = kAccRowThreads / 64;
constexpr int kAccRowHold = 4;                               // super-tiles per wave and pass of the row form
constexpr int kSuper = 1024;                                 // tokens per super-tile of the row form
constexpr int kAccSegThreads = 256;
constexpr int kAccSub = 256;                                 // tokens per sub-tile: one float4 per lane of a wave
constexpr int kAccSubPerWave = 4;                            // sub-tiles per wave and segment
constexpr int kAccSeg = kAccSegThreads / 64 * kAccSubPerWave * kAccSub;  // 4096 tokens per segment
constexpr int kAccThreads = 256;                             // (B)
constexpr int kAccRowsPerDraw = kAccThreads / 64;            // positions per workgroup of (B)

struct AccWork {
  double* sub;   // [B][nsub][parts] residual sums per sub-tile: one per 256 tokens (written by (A)) or four
                 // partial sums per 1024 tokens (written with r by the quadrature's evaluation), read by (B)
  int64_t nsub;  // sub-tiles per row
};
static_assert(kAccSub % 256 == 0 && kResSub % 256 == 0, "whole float4 per lane in a sub-tile's search");

// Row form: one workgroup per position (the residual and its mass not asked for).
template <bool kVec, bool kSel>
__global__ __launch_bounds__(kAccRowThreads) void accept_row_kernel(
    const float* __restrict__ p, const float* __restrict__ r, const int32_t* __restrict__ sel_token,
    const float* __restrict__ u, uint64_t seed, uint64_t offset, int64_t V, int32_t* __restrict__ out_token,
    uint8_t* __restrict__ accepted, int32_t* __restrict__ row_status, SelArgs sel) {
  extern __shared__ double s_tile[];  // one sum per super-tile
  __shared__ int s_bad;
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const float* pb = p + b * V;
  const float* rb = r + b * V;
  float uu[3];
  position_uniforms(u, seed, offset, b, uu);
  const Decision d = take_decision<kSel>(pb, rb, sel_token, sel, b, V, uu);
  if (kSel && tid == 0) {
    if (sel.sel_index) sel.sel_index[b] = d.istar;
    if (sel.sel_token) sel.sel_token[b] = d.Y;
    if (d.st && row_status) row_status[b] |= d.st;
  }
  if (d.acc || d.bad_y) {  // the same in every thread: the row is not read
    if (tid == 0) {
      out_token[b] = d.bad_y ? -1 : d.Y;
      accepted[b] = d.acc ? 1 : 0;
      if (d.bad_y && row_status) row_status[b] |= d.y_ok ? kRowBadProb : kRowBadDraft;
    }
    return;
  }
  if (tid == 0) s_bad = 0;
  __syncthreads();
  const int64_t nsuper = (V + kSuper - 1) / kSuper;
  int bad = 0;
  // kAccRowHold super-tiles per wave and pass, all of their row loads issued before any
  // arithmetic; the last pass's values stay in registers for the search below
  float pv[kAccRowHold][4][4], rv[kAccRowHold][4][4];
  for (int64_t st0 = wid; st0 < nsuper; st0 += kAccRowHold * kAccRowWaves) {
#pragma unroll
    for (int h = 0; h < kAccRowHold; ++h) {
      const int64_t st = st0 + h * kAccRowWaves;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t x0 = st * kSuper + 256 * k + 4 * lane;
        load4<kVec>(pb, x0, V, pv[h][k]);  // tokens at or past V (incl. a whole missing super-tile) read as 0
        load4<kVec>(rb, x0, V, rv[h][k]);
      }
    }
#pragma unroll
    for (int h = 0; h < kAccRowHold; ++h) {
      const int64_t st = st0 + h * kAccRowWaves;
      if (st >= nsuper) break;
      double local = 0.0;
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bad |= (int)(bad_prob(pv[h][k][i]) || bad_prob(rv[h][k][i]));
          local += residual_of(pv[h][k][i], rv[h][k][i]);
        }
      const double tot = wave_sum_dpp(local);
      if (lane == 0) s_tile[st] = tot;
    }
  }
  if (bad) atomicOr(&s_bad, 1);
  __syncthreads();
  // every wave: the totals and the prefix over the super-tiles (lane l takes a contiguous range)
  const bool row_bad = s_bad != 0;
  const int64_t per_lane = (nsuper + 63) / 64;
  const int64_t s_lo = lane * per_lane, s_hi = (s_lo + per_lane < nsuper) ? s_lo + per_lane : nsuper;
  double lane_sum = 0.0;
  for (int64_t s = s_lo; s < s_hi; ++s) lane_sum += s_tile[s];
  const double incl = wave_inclusive_scan_dpp(lane_sum, lane);
  const double Z = __shfl(incl, 63, 64);
  double excl = __shfl_up(incl, 1, 64);
  if (lane == 0) excl = 0.0;
  if (row_bad || !(Z > 0.0)) {
    if (wid == 0 && lane == 0) {
      out_token[b] = row_bad ? -1 : d.Y;
      accepted[b] = row_bad ? 0 : 1;
      if (row_status) row_status[b] |= row_bad ? kRowBadProb : kRowForced;
    }
    return;
  }
  const double thr = (double)uu[2] * Z;
  // first super-tile whose running sum exceeds thr
  int64_t my_st = -1;
  double my_prev = 0.0, run = excl;
  for (int64_t s = s_lo; s < s_hi; ++s) {
    const double prev = run;
    run += s_tile[s];
    if (run > thr) {
      my_st = s;
      my_prev = prev;
      break;
    }
  }
  const unsigned long long hit = __builtin_amdgcn_ballot_w64(my_st >= 0);
  int64_t st_star;
  double base;
  if (hit) {
    const int src = __ffsll((long long)hit) - 1;
    st_star = __shfl(my_st, src, 64);
    base = __shfl(my_prev, src, 64);
  } else {
    // rounding put u_res * Z at or past every running sum: the last super-tile with mass
    int64_t last = -1;
    for (int64_t s = s_lo; s < s_hi; ++s)
      if (s_tile[s] > 0.0) last = s;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t o = __shfl_xor(last, off, 64);
      last = o > last ? o : last;
    }
    st_star = last;
    base = thr;  // forces the in-tile search to its own fallback
  }
  if (st_star < 0) {  // unreachable with Z > 0; keeps every load in bounds
    if (wid == 0 && lane == 0) {
      out_token[b] = d.Y;
      accepted[b] = 1;
      if (row_status) row_status[b] |= kRowForced;
    }
    return;
  }
  // the wave whose registers hold super-tile st_star searches it; a super-tile of an
  // earlier pass (rows past 32768 tokens) is re-read by wave 0
  const int owner = (int)(st_star % kAccRowWaves);
  const int64_t own0 = owner + kAccRowHold * kAccRowWaves * ((nsuper - 1 - owner) / (kAccRowHold * kAccRowWaves));
  const int64_t hh = (st_star - own0) / kAccRowWaves;  // which of the owner's last-pass super-tiles
  const bool in_regs = st_star >= own0 && hh < kAccRowHold;
  if (wid != (in_regs ? owner : 0)) return;
  float ps[4][4], rs32[4][4];
  if (in_regs) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = pv[0][k][i], c = rv[0][k][i];
#pragma unroll
        for (int h = 1; h < kAccRowHold; ++h) {
          a = (hh == h) ? pv[h][k][i] : a;
          c = (hh == h) ? rv[h][k][i] : c;
        }
        ps[k][i] = a;
        rs32[k][i] = c;
      }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t x0 = st_star * kSuper + 256 * k + 4 * lane;
      load4<kVec>(pb, x0, V, ps[k]);
      load4<kVec>(rb, x0, V, rs32[k]);
    }
  }
  int64_t found = -1;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (found >= 0) break;  // uniform
    double rs[4], local = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      rs[i] = residual_of(ps[k][i], rs32[k][i]);
      local += rs[i];
    }
    const double li = wave_inclusive_scan_dpp(local, lane);
    double le = __shfl_up(li, 1, 64);
    if (lane == 0) le = 0.0;
    double c = base + le;
    int my = -1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c += rs[i];
      if (my < 0 && rs[i] > 0.0 && c > thr) my = i;
    }
    const unsigned long long h2 = __builtin_amdgcn_ballot_w64(my >= 0);
    if (h2) {
      const int src = __ffsll((long long)h2) - 1;
      found = st_star * kSuper + 256 * k + 4 * src + __shfl(my, src, 64);
    } else {
      base += __shfl(li, 63, 64);
    }
  }
  if (found < 0) {
    // fallback: the last token of the super-tile with a positive residual
    int64_t last = -1;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t x0 = st_star * kSuper + 256 * k + 4 * lane;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (x0 + i < V && residual_of(ps[k][i], rs32[k][i]) > 0.0) last = x0 + i;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t o = __shfl_xor(last, off, 64);
      last = o > last ? o : last;
    }
    found = last;
  }
  if (lane == 0) {
    out_token[b] = (int32_t)found;
    accepted[b] = 0;
  }
}

// Segment form (A).
template <bool kVec>
__global__ __launch_bounds__(kAccSegThreads) void accept_seg_kernel(const float* __restrict__ p,
                                                                    const float* __restrict__ r, int64_t V,
                                                                    float* __restrict__ residual, AccWork aw) {
  const int64_t b = blockIdx.y;
  const int64_t seg = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const float* pb = p + b * V;
  const float* rb = r + b * V;
  // the segment's sub-tiles: wave w takes kAccSubPerWave consecutive ones, all loads issued first
  const int64_t sub0 = seg * (kAccSeg / kAccSub) + wid * kAccSubPerWave;
  float pv[kAccSubPerWave][4], rv[kAccSubPerWave][4];
#pragma unroll
  for (int k = 0; k < kAccSubPerWave; ++k) {
    const int64_t x0 = (sub0 + k) * kAccSub + 4 * lane;
    load4<kVec>(pb, x0, V, pv[k]);  // tokens at or past V read as 0
    load4<kVec>(rb, x0, V, rv[k]);
  }
  float* resb = residual ? residual + b * V : nullptr;
  double sums[kAccSubPerWave];
#pragma unroll
  for (int k = 0; k < kAccSubPerWave; ++k) {
    const int64_t x0 = (sub0 + k) * kAccSub + 4 * lane;
    float rs[4];
    double local = 0.0;
    bool bad = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bad |= bad_prob(pv[k][i]) || bad_prob(rv[k][i]);
      const double dd = residual_of(pv[k][i], rv[k][i]);
      rs[i] = (float)dd;
      local += dd;
    }
    if (resb && x0 < V) {
      if (kVec && x0 + 3 < V) {
        typedef float f32x4v __attribute__((ext_vector_type(4)));
        const f32x4v v = {rs[0], rs[1], rs[2], rs[3]};
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4v*>(resb + x0));
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (x0 + i < V) resb[x0 + i] = rs[i];
      }
    }
    const double tot = wave_sum_dpp(local);
    sums[k] = (__builtin_amdgcn_ballot_w64(bad) != 0) ? (double)NAN : tot;
  }
  double v = sums[0];
#pragma unroll
  for (int k = 1; k < kAccSubPerWave; ++k) v = (lane == k) ? sums[k] : v;
  if (lane < kAccSubPerWave && sub0 + lane < aw.nsub) aw.sub[b * aw.nsub + sub0 + lane] = v;
}

// Segment form (B): one wave per position (the body is draw_from_sums).
template <bool kVec, bool kSel, int kParts, int kSub>
__global__ __launch_bounds__(kAccThreads) void accept_draw_kernel(
    const float* __restrict__ p, const float* __restrict__ r, const int32_t* __restrict__ sel_token,
    const float* __restrict__ u, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
    int32_t* __restrict__ out_token, uint8_t* __restrict__ accepted, double* __restrict__ residual_mass,
    int32_t* __restrict__ row_status, SelArgs sel, AccWork aw) {
  const int lane = threadIdx.x & 63;
  const int64_t b = (int64_t)blockIdx.x * kAccRowsPerDraw + (threadIdx.x >> 6);
  if (b >= B) return;
  draw_from_sums<kVec, kSel, kParts, kSub>(p + b * V, r + b * V, aw.sub + b * aw.nsub * kParts, aw.nsub, sel_token,
                                           u, seed, offset, b, V, lane, out_token, accepted, residual_mass,
                                           row_status, sel);
}

}  // namespace

hipError_t launch_select(const float* p, const float* q, const int32_t* drafts, const float* u, uint64_t seed,
                         uint64_t offset, int64_t B, int64_t V, int K, int32_t* sel_index, int32_t* sel_token,
                         int32_t* row_status, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, st, p, q, nullptr, drafts, u,
                     seed, offset, B, V, K, sel_index, sel_token, row_status);
  return hipGetLastError();
}

hipError_t launch_select_successive(const float* p, const float* q, const float* r_stages, const int32_t* drafts,
                                    const float* u_sel, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int K,
                                    int32_t* sel_index, int32_t* sel_token, int32_t* row_status, hipStream_t st) {
  hipLaunchKernelGGL(select_successive_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, st, p, q, r_stages,
                     drafts, u_sel, seed, offset, B, V, K, sel_index, sel_token, row_status);
  return hipGetLastError();
}

hipError_t launch_select_pair(const float* p, const float* q1, const float* q2, const int32_t* drafts,
                              const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                              int32_t* sel_index, int32_t* sel_token, int32_t* row_status, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, st, p, q1, q2, drafts, u, seed,
                     offset, B, V, 2, sel_index, sel_token, row_status);
  return hipGetLastError();
}

namespace {

size_t align256_acc(size_t x) { return (x + 255) / 256 * 256; }

template <bool kSel>
hipError_t launch_accept_impl(const float* p, const float* r, const int32_t* sel_token, const float* u,
                              uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t* out_token,
                              uint8_t* accepted, float* residual, double* residual_mass, int32_t* row_status,
                              const SelArgs& sel, void* workspace, hipStream_t st) {
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(r) |
                                     reinterpret_cast<uintptr_t>(residual)) % 16 == 0);
  if (residual == nullptr && residual_mass == nullptr) {  // row form: only rejected positions read their rows
    const size_t lds = sizeof(double) * (size_t)((V + kSuper - 1) / kSuper);
    if (vec) {
      hipLaunchKernelGGL((accept_row_kernel<true, kSel>), dim3((unsigned)B), dim3(kAccRowThreads), lds, st, p, r,
                         sel_token, u, seed, offset, V, out_token, accepted, row_status, sel);
    } else {
      hipLaunchKernelGGL((accept_row_kernel<false, kSel>), dim3((unsigned)B), dim3(kAccRowThreads), lds, st, p, r,
                         sel_token, u, seed, offset, V, out_token, accepted, row_status, sel);
    }
    return hipGetLastError();
  }
  AccWork aw;
  aw.sub = static_cast<double*>(workspace);
  aw.nsub = (V + kAccSub - 1) / kAccSub;
  const int64_t nseg = (V + kAccSeg - 1) / kAccSeg;
  const dim3 ga((unsigned)nseg, (unsigned)B);
  const dim3 gb((unsigned)((B + kAccRowsPerDraw - 1) / kAccRowsPerDraw));
  if (vec) {
    hipLaunchKernelGGL((accept_seg_kernel<true>), ga, dim3(kAccSegThreads), 0, st, p, r, V, residual, aw);
    hipLaunchKernelGGL((accept_draw_kernel<true, kSel, 1, kAccSub>), gb, dim3(kAccThreads), 0, st, p, r, sel_token, u, seed,
                       offset, B, V, out_token, accepted, residual_mass, row_status, sel, aw);
  } else {
    hipLaunchKernelGGL((accept_seg_kernel<false>), ga, dim3(kAccSegThreads), 0, st, p, r, V, residual, aw);
    hipLaunchKernelGGL((accept_draw_kernel<false, kSel, 1, kAccSub>), gb, dim3(kAccThreads), 0, st, p, r, sel_token, u, seed,
                       offset, B, V, out_token, accepted, residual_mass, row_status, sel, aw);
  }
  return hipGetLastError();
}

}  // namespace

size_t workspace_bytes_accept(int64_t B, int64_t V) {
  const int64_t n1 = (V + kAccSub - 1) / kAccSub, n4 = (V + kResSub - 1) / kResSub;  // the two layouts
  return align256_acc(sizeof(double) * (size_t)(B * std::max(n1, n4 * kResParts)));
}

// Selection and Algorithm 1 from the residual sums the quadrature's evaluation wrote
// with r (four partial sums per 1024-token sub-tile): the segment form's (B) alone.
hipError_t launch_select_accept_sums(const float* p, const float* q, const float* q2, const float* r,
                                     const int32_t* drafts, const float* u, uint64_t seed, uint64_t offset,
                                     int64_t B, int64_t V, int K, int32_t* sel_index, int32_t* sel_token,
                                     int32_t* out_token, uint8_t* accepted, double* residual_mass,
                                     int32_t* row_status, void* workspace, hipStream_t st) {
  const SelArgs sel = {q, q2, drafts, K, sel_index, sel_token};
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(r)) % 16 == 0);
  AccWork aw;
  aw.sub = static_cast<double*>(workspace);
  aw.nsub = (V + kResSub - 1) / kResSub;
  const dim3 gb((unsigned)((B + kAccRowsPerDraw - 1) / kAccRowsPerDraw));
  if (vec)
    hipLaunchKernelGGL((accept_draw_kernel<true, true, kResParts, kResSub>), gb, dim3(kAccThreads), 0, st, p, r, nullptr, u,
                       seed, offset, B, V, out_token, accepted, residual_mass, row_status, sel, aw);
  else
    hipLaunchKernelGGL((accept_draw_kernel<false, true, kResParts, kResSub>), gb, dim3(kAccThreads), 0, st, p, r, nullptr, u,
                       seed, offset, B, V, out_token, accepted, residual_mass, row_status, sel, aw);
  return hipGetLastError();
}

hipError_t launch_accept(const float* p, const float* r, const int32_t* sel_token, const float* u, uint64_t seed,
                         uint64_t offset, int64_t B, int64_t V, int32_t* out_token, uint8_t* accepted,
                         float* residual, double* residual_mass, int32_t* row_status, void* workspace,
                         hipStream_t st) {
  const SelArgs none = {nullptr, nullptr, nullptr, 0, nullptr, nullptr};
  return launch_accept_impl<false>(p, r, sel_token, u, seed, offset, B, V, out_token, accepted, residual,
                                   residual_mass, row_status, none, workspace, st);
}

hipError_t launch_select_accept(const float* p, const float* q, const float* q2, const float* r,
                                const int32_t* drafts, const float* u, uint64_t seed, uint64_t offset, int64_t B,
                                int64_t V, int K, int32_t* sel_index, int32_t* sel_token, int32_t* out_token,
                                uint8_t* accepted, float* residual, double* residual_mass, int32_t* row_status,
                                void* workspace, hipStream_t st) {
  const SelArgs sel = {q, q2, drafts, K, sel_index, sel_token};
  return launch_accept_impl<true>(p, r, nullptr, u, seed, offset, B, V, out_token, accepted, residual,
                                  residual_mass, row_status, sel, workspace, st);
}

}  // namespace mdss
