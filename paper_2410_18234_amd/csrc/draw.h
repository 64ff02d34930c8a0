// Selection of the intermediate token (Definition 1, index form with the classical
// weights) and the draw of Algorithm 1 from residual sums: device code shared by the
// sampling kernels and the top-s quadrature's fused step.
#pragma once

#include "common.h"

#include <math.h>

namespace mdss {

namespace {

// Weight of one draft (fp64 p(x)/q(x), the classical weight of Definition 1);
// an invalid draft (outside [0, V), q(x) = 0, or a NaN/negative/inf p or q)
// adds its status bit and weighs 0.
__device__ __forceinline__ double draft_weight(bool in_range, float pv, float qv, int& st) {
  // branch-free (selects), so that a caller's per-draft arrays stay in place
  const bool badp = bad_prob(pv) || bad_prob(qv);
  const bool zq = !(qv > 0.0f);
  st |= !in_range ? kRowBadDraft : (badp ? kRowBadProb : (zq ? kRowBadDraft : 0));
  const double w = (double)pv / (double)qv;
  return (in_range && !badp && !zq) ? w : 0.0;
}

// Selected index from the weights: W = sum_i w_i left to right, the smallest i
// with u_sel * W < w_1 + ... + w_i; floor(u_sel K) when W = 0.
__device__ __forceinline__ int select_index(const double* w, int K, double us) {
  double W = 0.0;
  for (int i = 0; i < K; ++i) W += w[i];
  int istar = K - 1;
  if (W > 0.0) {
    const double t = us * W;
    double C = 0.0;
    for (int i = 0; i < K; ++i) {
      C += w[i];
      if (t < C) {
        istar = i;
        break;
      }
    }
  } else {
    istar = (int)floor(us * (double)K);
  }
  return istar < 0 ? 0 : (istar >= K ? K - 1 : istar);  // only a uniform outside [0, 1) can leave the range
}

template <bool kVec>
__device__ __forceinline__ void load4(const float* __restrict__ a, int64_t x0, int64_t V, float v[4]) {
  if (kVec && x0 + 3 < V) {
    const float4 t = *reinterpret_cast<const float4*>(a + x0);
    v[0] = t.x;
    v[1] = t.y;
    v[2] = t.z;
    v[3] = t.w;
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (x0 + i < V) ? a[x0 + i] : 0.0f;
  }
}

// Selection arguments of the fused form (selection and Algorithm 1 in one
// call): drafts [B][K], q (and q2 for two drafts from different
// distributions), and the selection outputs (each nullable).
struct SelArgs {
  const float* q;
  const float* q2;
  const int32_t* drafts;
  int K;
  int32_t* sel_index;
  int32_t* sel_token;
};

// The selection of the intermediate token (fused form: from the drafts, with
// p, q and r of every draft read at once, so p(Y) and r(Y) come with them) or the
// given selected token, and the accept test u_acc r(Y) < p(Y) in fp64.
struct Decision {
  int32_t Y;      // selected token (-1 if the drafts are invalid)
  int32_t istar;  // selected index (fused form)
  int st;         // status bits of the selection
  bool y_ok, bad_y, acc;
};

template <bool kSel>
__device__ __forceinline__ Decision take_decision(const float* __restrict__ pb, const float* __restrict__ rb,
                                                  const int32_t* __restrict__ sel_token, const SelArgs& sel,
                                                  int64_t b, int64_t V, const float (&uu)[3]) {
  Decision d;
  d.st = 0;
  d.istar = -1;
  float pY = 0.0f, rY = 0.0f;
  if (kSel) {
    int32_t x[kMaxK];
    float pv[kMaxK], qv[kMaxK], rv[kMaxK];
    bool in[kMaxK];
    // the drafts past K are skipped by branches on K (the same in every lane)
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      x[i] = -1;
      if (i < sel.K) x[i] = sel.drafts[b * sel.K + i];
      in[i] = x[i] >= 0 && (int64_t)x[i] < V;
    }
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      pv[i] = qv[i] = rv[i] = 0.0f;
      if (i < sel.K) {
        const float* qi = (sel.q2 != nullptr && i == 1) ? sel.q2 : sel.q;
        pv[i] = in[i] ? pb[x[i]] : 0.0f;
        qv[i] = in[i] ? qi[b * V + x[i]] : 0.0f;
        rv[i] = in[i] ? rb[x[i]] : 0.0f;
      }
    }
    double w[kMaxK];
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      w[i] = 0.0;
      if (i < sel.K) w[i] = draft_weight(in[i], pv[i], qv[i], d.st);
    }
    d.istar = d.st ? -1 : select_index(w, sel.K, (double)uu[0]);
    d.Y = -1;
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      if (i == d.istar) {
        d.Y = x[i];
        pY = pv[i];
        rY = rv[i];
      }
    }
  } else {
    d.Y = sel_token[b];
    if (d.Y >= 0 && (int64_t)d.Y < V) {
      pY = pb[d.Y];
      rY = rb[d.Y];
    }
  }
  d.y_ok = (d.Y >= 0) && ((int64_t)d.Y < V);
  d.bad_y = !d.y_ok || bad_prob(pY) || bad_prob(rY);
  d.acc = !d.bad_y && ((double)uu[1] * (double)rY < (double)pY);
  return d;
}

// Selection (kSel: from the drafts) and Algorithm 1 for position b by one wave (lane =
// its lane), with Z and the running sums from kParts partial residual sums per
// kSub-token sub-tile (sb: the row's [nsub][kParts], added in order; in global or
// LDS memory).  pb, rb: the row's p and r.  Writes out_token[b], accepted[b],
// residual_mass[b] (nullable), the selection outputs, and ORs flags into row_status[b].
template <bool kVec, bool kSel, int kParts, int kSub>
__device__ __forceinline__ void draw_from_sums(const float* __restrict__ pb, const float* __restrict__ rb,
                                               const double* sb, int64_t nsub, const int32_t* __restrict__ sel_token,
                                               const float* __restrict__ u, uint64_t seed, uint64_t offset,
                                               int64_t b, int64_t V, int lane, int32_t* __restrict__ out_token,
                                               uint8_t* __restrict__ accepted, double* __restrict__ residual_mass,
                                               int32_t* __restrict__ row_status, const SelArgs& sel) {
  const auto sub_at = [&](int64_t s) -> double {  // the residual sum of sub-tile s
    double v = sb[s * kParts];
#pragma unroll
    for (int k = 1; k < kParts; ++k) v += sb[s * kParts + k];
    return v;
  };
  // Z and the running sums: lane l takes the sub-tiles [l per, (l + 1) per), in order,
  // read together with the decision's loads
  const int64_t per = (nsub + 63) / 64;
  const int64_t s_lo = lane * per, s_hi = (s_lo + per < nsub) ? s_lo + per : nsub;
  double lane_sum = 0.0;
  for (int64_t s = s_lo; s < s_hi; ++s) lane_sum += sub_at(s);
  float uu[3];
  position_uniforms(u, seed, offset, b, uu);
  const Decision d = take_decision<kSel>(pb, rb, sel_token, sel, b, V, uu);
  if (kSel && lane == 0) {
    if (sel.sel_index) sel.sel_index[b] = d.istar;
    if (sel.sel_token) sel.sel_token[b] = d.Y;
    if (d.st && row_status) row_status[b] |= d.st;
  }
  const int32_t Y = d.Y;
  const bool acc = d.acc, bad_y = d.bad_y, y_ok = d.y_ok;
  const bool row_bad = __builtin_amdgcn_ballot_w64(lane_sum != lane_sum) != 0;  // a NaN sub-tile sum
  const double incl = wave_inclusive_scan_dpp(lane_sum, lane);
  const double Z = __shfl(incl, 63, 64);
  double excl = __shfl_up(incl, 1, 64);  // the running sum before this lane's sub-tiles
  if (lane == 0) excl = 0.0;
  if (lane == 0 && residual_mass) residual_mass[b] = row_bad ? (double)NAN : Z;
  if (row_bad || bad_y) {
    if (lane == 0) {
      out_token[b] = -1;
      accepted[b] = 0;
      if (row_status) row_status[b] |= (row_bad || y_ok) ? kRowBadProb : kRowBadDraft;
    }
    return;
  }
  if (acc) {
    if (lane == 0) {
      out_token[b] = Y;
      accepted[b] = 1;
    }
    return;
  }
  if (!(Z > 0.0)) {
    if (lane == 0) {
      out_token[b] = Y;
      accepted[b] = 1;
      if (row_status) row_status[b] |= kRowForced;
    }
    return;
  }
  const double thr = (double)uu[2] * Z;
  // first sub-tile whose running sum exceeds thr
  int64_t my_s = -1;
  double my_prev = 0.0, run = excl;
  for (int64_t s = s_lo; s < s_hi; ++s) {
    const double prev = run;
    run += sub_at(s);
    if (run > thr) {
      my_s = s;
      my_prev = prev;
      break;
    }
  }
  const unsigned long long hit = __builtin_amdgcn_ballot_w64(my_s >= 0);
  int64_t s_star;
  double base;
  if (hit) {
    const int src = __ffsll((long long)hit) - 1;
    s_star = __shfl(my_s, src, 64);
    base = __shfl(my_prev, src, 64);
  } else {
    // rounding put u_res * Z at or past every running sum: the last sub-tile with mass
    int64_t last = -1;
    for (int64_t s = s_lo; s < s_hi; ++s)
      if (sub_at(s) > 0.0) last = s;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t o = __shfl_xor(last, off, 64);
      last = o > last ? o : last;
    }
    s_star = last;
    base = thr;  // forces the in-tile search to its own fallback
  }
  if (s_star < 0) {  // unreachable with Z > 0; keeps every load in bounds
    if (lane == 0) {
      out_token[b] = Y;
      accepted[b] = 1;
      if (row_status) row_status[b] |= kRowForced;
    }
    return;
  }
  // the token inside sub-tile s_star: kPer consecutive entries per lane, lane prefix, then the lane's own entries
  constexpr int kPer = kSub / 64;
  const int64_t x0 = s_star * kSub + kPer * lane;
  float pv[kPer], rv[kPer];
#pragma unroll
  for (int j = 0; j < kPer; j += 4) {
    load4<kVec>(pb, x0 + j, V, pv + j);
    load4<kVec>(rb, x0 + j, V, rv + j);
  }
  double rs[kPer], local = 0.0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    rs[i] = residual_of(pv[i], rv[i]);
    local += rs[i];
  }
  const double li = wave_inclusive_scan_dpp(local, lane);
  double le = __shfl_up(li, 1, 64);
  if (lane == 0) le = 0.0;
  double c = base + le;
  int my = -1;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    c += rs[i];
    if (my < 0 && rs[i] > 0.0 && c > thr) my = i;
  }
  const unsigned long long h2 = __builtin_amdgcn_ballot_w64(my >= 0);
  int64_t found;
  if (h2) {
    const int src = __ffsll((long long)h2) - 1;
    found = s_star * kSub + kPer * src + __shfl(my, src, 64);
  } else {
    // fallback: the last token of the sub-tile with a positive residual
    int64_t last = -1;
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (x0 + i < V && rs[i] > 0.0) last = x0 + i;
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


}  // namespace

}  // namespace mdss
