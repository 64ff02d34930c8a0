// Selection of the intermediate token (Definition 1, index form with the
// classical weights) and single-draft speculative sampling of that token
// against the target (Algorithm 1), gfx950.
//
// Notation: p = target, q = draft, r = induced distribution of the selected
// token (the proposal of Algorithm 1).  Decisions are taken in fp64 with the
// uniforms as 24-bit dyadics, so the accept test u * r(Y) < p(Y) is exact.
#include "common.h"

#include <math.h>

namespace mdss {

namespace {

// ------------------------------------------------------------------ selection
// Weight of one draft (fp64 p(x)/q(x), the classical weight of Definition 1);
// an invalid draft (outside [0, V), q(x) = 0, or a NaN/negative/inf p or q)
// adds its status bit and weighs 0.
__device__ __forceinline__ double draft_weight(bool in_range, float pv, float qv, int& st) {
  if (!in_range) {
    st |= kRowBadDraft;
    return 0.0;
  }
  if (bad_prob(pv) || bad_prob(qv)) {
    st |= kRowBadProb;
    return 0.0;
  }
  if (!(qv > 0.0f)) {
    st |= kRowBadDraft;
    return 0.0;
  }
  return (double)pv / (double)qv;
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
// One workgroup of 16 waves per position.  Pass 1 streams the row in
// super-tiles of 1024 tokens (wave w takes super-tiles w, w+16, ...), forms
// res = max(0, p - r) in fp64, optionally stores it, and keeps each
// super-tile's sum in LDS.  Wave 0 then scans the super-tile sums, finds the
// super-tile where the running sum first exceeds u_res * Z and re-reads only
// that one (four 256-token sub-tiles, each a lane scan) to locate the token.
constexpr int kAccThreads = 1024;
constexpr int kAccWaves = kAccThreads / 64;
constexpr int kSuper = 1024;

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

__device__ __forceinline__ double residual_of(float pv, float rv) {
  const double d = (double)pv - (double)rv;
  return d > 0.0 ? d : 0.0;
}

// Selection arguments of the fused form (selection and Algorithm 1 in one
// launch): drafts [B][K], q (and q2 for two drafts from different
// distributions), and the selection outputs (each nullable).
struct SelArgs {
  const float* q;
  const float* q2;
  const int32_t* drafts;
  int K;
  int32_t* sel_index;
  int32_t* sel_token;
};

template <bool kVec, bool kSel>
__global__ __launch_bounds__(kAccThreads) void accept_kernel(
    const float* __restrict__ p, const float* __restrict__ r, const int32_t* __restrict__ sel_token,
    const float* __restrict__ u, uint64_t seed, uint64_t offset, int64_t V, int32_t* __restrict__ out_token,
    uint8_t* __restrict__ accepted, float* __restrict__ residual, double* __restrict__ residual_mass,
    int32_t* __restrict__ row_status, SelArgs sel) {
  extern __shared__ double s_tile[];  // one sum per super-tile
  __shared__ int s_bad;
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const float* pb = p + b * V;
  const float* rb = r + b * V;
  float uu[3];
  position_uniforms(u, seed, offset, b, uu);
  int32_t Y;
  float pY = 0.0f, rY = 0.0f;
  if (kSel) {
    // the selection of the intermediate token, with p, q and r of every draft
    // read at once (Y is one of the drafts, so p(Y) and r(Y) come with them)
    int32_t x[kMaxK];
    float pv[kMaxK], qv[kMaxK], rv[kMaxK];
    bool in[kMaxK];
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      x[i] = i < sel.K ? sel.drafts[b * sel.K + i] : -1;
      in[i] = x[i] >= 0 && (int64_t)x[i] < V;
    }
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      const float* qi = (sel.q2 != nullptr && i == 1) ? sel.q2 : sel.q;
      pv[i] = in[i] ? pb[x[i]] : 0.0f;
      qv[i] = in[i] ? qi[b * V + x[i]] : 0.0f;
      rv[i] = in[i] ? rb[x[i]] : 0.0f;
    }
    int st = 0;
    double w[kMaxK];
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) w[i] = i < sel.K ? draft_weight(in[i], pv[i], qv[i], st) : 0.0;
    const int istar = st ? -1 : select_index(w, sel.K, (double)uu[0]);
    Y = -1;
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      if (i == istar) {
        Y = x[i];
        pY = pv[i];
        rY = rv[i];
      }
    }
    if (tid == 0) {
      if (sel.sel_index) sel.sel_index[b] = istar;
      if (sel.sel_token) sel.sel_token[b] = Y;
      if (st && row_status) row_status[b] |= st;
    }
  } else {
    Y = sel_token[b];
    if (Y >= 0 && (int64_t)Y < V) {
      pY = pb[Y];
      rY = rb[Y];
    }
  }
  const bool y_ok = (Y >= 0) && ((int64_t)Y < V);
  const bool bad_y = !y_ok || bad_prob(pY) || bad_prob(rY);
  const bool acc = !bad_y && ((double)uu[1] * (double)rY < (double)pY);
  const bool need_pass = (residual != nullptr) || (residual_mass != nullptr) || (!acc && !bad_y);
  if (!need_pass) {
    if (tid == 0) {
      out_token[b] = bad_y ? -1 : Y;
      accepted[b] = acc ? 1 : 0;
      if (bad_y && row_status) row_status[b] |= y_ok ? kRowBadProb : kRowBadDraft;
    }
    return;
  }
  if (tid == 0) s_bad = 0;
  __syncthreads();
  const int64_t nsuper = (V + kSuper - 1) / kSuper;
  float* resb = residual ? residual + b * V : nullptr;
  int bad = 0;
  // two super-tiles per wave and iteration: all 16 row loads are issued before any arithmetic
  for (int64_t st0 = wid; st0 < nsuper; st0 += 2 * kAccWaves) {
    float pv[2][4][4], rv[2][4][4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t st = st0 + h * kAccWaves;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t x0 = st * kSuper + 256 * k + 4 * lane;
        load4<kVec>(pb, x0, V, pv[h][k]);  // tokens at or past V (incl. a whole missing super-tile) read as 0
        load4<kVec>(rb, x0, V, rv[h][k]);
      }
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t st = st0 + h * kAccWaves;
      if (st >= nsuper) break;
      double local = 0.0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t x0 = st * kSuper + 256 * k + 4 * lane;
        float rs[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bad |= (int)(bad_prob(pv[h][k][i]) || bad_prob(rv[h][k][i]));
          const double d = residual_of(pv[h][k][i], rv[h][k][i]);
          rs[i] = (float)d;
          local += d;
        }
        if (resb) {
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
      }
      const double tot = wave_sum(local);
      if (lane == 0) s_tile[st] = tot;
    }
  }
  if (bad) atomicOr(&s_bad, 1);
  __syncthreads();
  if (wid != 0) return;

  // wave 0: totals, prefix over super-tiles, draw
  const bool row_bad = s_bad != 0;
  const int64_t per_lane = (nsuper + 63) / 64;
  const int64_t s_lo = lane * per_lane, s_hi = (s_lo + per_lane < nsuper) ? s_lo + per_lane : nsuper;
  double lane_sum = 0.0;
  for (int64_t s = s_lo; s < s_hi; ++s) lane_sum += s_tile[s];
  const double incl = wave_inclusive_scan(lane_sum, lane);
  const double Z = __shfl(incl, 63, 64);
  double excl = __shfl_up(incl, 1, 64);
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
  const unsigned long long hit = __ballot(my_st >= 0);
  int64_t st_star;
  double prev_star;
  if (hit) {
    const int src = __ffsll((long long)hit) - 1;
    st_star = __shfl(my_st, src, 64);
    prev_star = __shfl(my_prev, src, 64);
  } else {
    // rounding put u_res * Z at or past every running sum: last super-tile with mass
    int64_t last = -1;
    for (int64_t s = s_lo; s < s_hi; ++s)
      if (s_tile[s] > 0.0) last = s;
    int64_t m = last;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t o = __shfl_xor(m, off, 64);
      m = o > m ? o : m;
    }
    st_star = m;
    prev_star = thr;  // forces the in-tile search to its own fallback
  }
  if (st_star < 0) {  // unreachable with Z > 0; keeps every load in bounds
    if (lane == 0) {
      out_token[b] = Y;
      accepted[b] = 1;
      if (row_status) row_status[b] |= kRowForced;
    }
    return;
  }
  // locate the token inside super-tile st_star (its four sub-tiles loaded at once)
  double base = prev_star;
  int32_t found = -1;
  float pvs[4][4], rvs[4][4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t x0 = st_star * kSuper + 256 * k + 4 * lane;
    load4<kVec>(pb, x0, V, pvs[k]);
    load4<kVec>(rb, x0, V, rvs[k]);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (found >= 0) break;  // uniform
    double rs[4], local = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      rs[i] = residual_of(pvs[k][i], rvs[k][i]);
      local += rs[i];
    }
    const double li = wave_inclusive_scan(local, lane);
    double le = __shfl_up(li, 1, 64);
    if (lane == 0) le = 0.0;
    double c = base + le;
    int my = -1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c += rs[i];
      if (my < 0 && rs[i] > 0.0 && c > thr) my = i;
    }
    const unsigned long long h2 = __ballot(my >= 0);
    if (h2) {
      const int src = __ffsll((long long)h2) - 1;
      const int mi = __shfl(my, src, 64);
      found = (int32_t)(st_star * kSuper + 256 * k + 4 * src + mi);
    } else {
      base += __shfl(li, 63, 64);
    }
  }
  if (found < 0) {
    // fallback: last token of the super-tile with positive residual
    int64_t last = -1;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t x0 = st_star * kSuper + 256 * k + 4 * lane;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (x0 + i < V && residual_of(pvs[k][i], rvs[k][i]) > 0.0) last = x0 + i;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t o = __shfl_xor(last, off, 64);
      last = o > last ? o : last;
    }
    found = (int32_t)last;
  }
  if (lane == 0) {
    out_token[b] = found;
    accepted[b] = 0;
  }
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

template <bool kSel>
hipError_t launch_accept_impl(const float* p, const float* r, const int32_t* sel_token, const float* u,
                              uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t* out_token,
                              uint8_t* accepted, float* residual, double* residual_mass, int32_t* row_status,
                              const SelArgs& sel, hipStream_t st) {
  const int64_t nsuper = (V + kSuper - 1) / kSuper;
  const size_t lds = sizeof(double) * (size_t)nsuper;
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(r) |
                                     reinterpret_cast<uintptr_t>(residual)) % 16 == 0);
  if (vec) {
    hipLaunchKernelGGL((accept_kernel<true, kSel>), dim3((unsigned)B), dim3(kAccThreads), lds, st, p, r, sel_token, u,
                       seed, offset, V, out_token, accepted, residual, residual_mass, row_status, sel);
  } else {
    hipLaunchKernelGGL((accept_kernel<false, kSel>), dim3((unsigned)B), dim3(kAccThreads), lds, st, p, r, sel_token,
                       u, seed, offset, V, out_token, accepted, residual, residual_mass, row_status, sel);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_accept(const float* p, const float* r, const int32_t* sel_token, const float* u, uint64_t seed,
                         uint64_t offset, int64_t B, int64_t V, int32_t* out_token, uint8_t* accepted,
                         float* residual, double* residual_mass, int32_t* row_status, hipStream_t st) {
  const SelArgs none = {nullptr, nullptr, nullptr, 0, nullptr, nullptr};
  return launch_accept_impl<false>(p, r, sel_token, u, seed, offset, B, V, out_token, accepted, residual,
                                   residual_mass, row_status, none, st);
}

hipError_t launch_select_accept(const float* p, const float* q, const float* q2, const float* r,
                                const int32_t* drafts, const float* u, uint64_t seed, uint64_t offset, int64_t B,
                                int64_t V, int K, int32_t* sel_index, int32_t* sel_token, int32_t* out_token,
                                uint8_t* accepted, float* residual, double* residual_mass, int32_t* row_status,
                                hipStream_t st) {
  const SelArgs sel = {q, q2, drafts, K, sel_index, sel_token};
  return launch_accept_impl<true>(p, r, nullptr, u, seed, offset, B, V, out_token, accepted, residual,
                                  residual_mass, row_status, sel, st);
}

}  // namespace mdss
