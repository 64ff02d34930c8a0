// Induced distribution r by an exponential-sum quadrature of the pair kernel.
//
// Notation: p = target, q = draft, w = p / q.  With the classical weights the
// selected-token law (proof of Theorem 1, eq. Ind; for K = 2 the pair form
// eq. p_Ieq0) is, for q(y) > 0 and p(y) > 0,
//   K i.i.d. drafts:  r(y) = K p(y) sum_{x_2..x_K in supp q} prod_j q(x_j) / (w(y) + sum_j w(x_j)),
//   two draft laws:   r(y) = p(y) [ sum_x q2(x) / (w1(y) + w2(x)) + sum_x q1(x) / (w1(x) + w2(y)) ],
// plus the closed forms of the zero-weight tokens.  Every denominator D is a
// sum of positive weights, and for D > 0
//   1 / D = integral over t in R of exp(t - D e^t) dt      (substitute s = D e^t),
// so with S(a) = sum_x q(x) exp(-a w(x)) the K-draft sum is
//   integral of exp(t) exp(-e^t w(y)) S(e^t)^(K-1) dt,
// and the pair sums factor the same way.  The trapezoidal rule on the grid
// t_k = k h turns the O(n^K) sum into O(n) work per node:
//   moments    S_k = sum_x q(x) exp(-a_k w(x)),   a_k = e^(t_k),
//   evaluation r(y) = p(y) sum_k c_k exp(-a_k w(y)),  c_k = K h a_k S_k^(K-1).
// Error of the rule (relative, for every D, independently of D): by Poisson
// summation the integrand exp(t - D e^t) has Fourier transform
// D^(-1+iv) Gamma(1 - iv), so the step-h sum differs from 1/D by at most
// 2 sum_{m>=1} |Gamma(1 + 2 pi i m / h)| / D, 4.8e-8 for h = 1/2.  The grid is
// cut where the left tail (t < t_lo: relative D e^t_lo) and the right tail
// (t > t_hi: relative exp(-D e^t_hi)) are below 1e-8 for every denominator of
// the row.  Every term is positive, so these relative bounds hold for the
// sums and for r; fp32 evaluation adds a few 1e-8.  A row's node count is
// (ln(D_max / D_min) + 21.3) / h: about 60 for LLM-like rows.
//
// Weights are scaled by a power of two per row (w' = w 2^sigma, the scale
// undone in r); rows whose positive weights span more than kEsWideRange
// binary exponents run the same kernels in fp64 (node parameters outside the
// fp32 range).  Decisions and closed forms are as in the pairwise kernels:
// zero-weight tokens (p = 0 < q) enter in closed form, a flagged row gets NaN.
#include "common.h"

#include <math.h>

#include <algorithm>

namespace mdss {

namespace {

constexpr int kEsThreads = 256;
constexpr int kEsMomPer = 16;                           // tokens per thread, moments pass
constexpr int kEsMomTile = kEsThreads * kEsMomPer;      // 4096 tokens per moments workgroup
constexpr int kEsEvalPer = 8;                           // tokens per thread, evaluation pass
constexpr int kEsEvalTile = kEsThreads * kEsEvalPer;    // 2048 tokens per evaluation workgroup
constexpr int kEsNB = 16;                               // nodes per unrolled block
constexpr int kEsMaxNodes = 480;                        // nodes of a row whose weights span <= 2^310
constexpr double kEsStep = 0.5;                         // h
constexpr double kEsLnEps = -18.420680743952367;        // ln 1e-8: left-tail cut
constexpr double kEsLnLnInvEps = 2.9134941423228814;    // ln ln 1e8: right-tail cut
constexpr double kEsLog2e = 1.4426950408889634;
constexpr int kEsWideRange = 180;  // binary exponent range of the weights above which fp64 is used

// Per (row, moments tile, law): statistics of the positive weights.
struct alignas(32) EsTileStat {
  double wmin;   // smallest positive weight, fp64 ratio (+inf if none)
  double wmax;   // largest weight (0 if none)
  int32_t npos;  // tokens with p > 0 and q > 0
  int32_t bad;   // a NaN, negative or infinite probability was read
  double q0;     // draft mass of zero-weight tokens (q > 0 = p)
};

// Per row: the evaluation plan.
struct alignas(64) EsPlan {
  int32_t flags;  // row status bits; a flagged row gets r = NaN
  int32_t k_lo;   // first node index: t_k = (k_lo + k) h
  int32_t nk;     // nodes (0: no quadrature term in this row)
  int32_t sigma;  // weight scale: w' = w 2^sigma
  int32_t wide;   // 1: nodes evaluated in fp64
  int32_t w64;    // 1: some weight p/q leaves the fp32 normal range: ratios taken in fp64
  int32_t pad[2];
  double q0[2];   // per law: draft mass of zero-weight tokens
  double pad2[2];
};

struct EsWork {
  EsTileStat* stat;  // [B][T1][L]
  EsPlan* plan;      // [B]
  float* beta;       // [B][kEsMaxNodes] fp32 node rates a_k log2(e) (scaled weights)
  double* alpha;     // [B][kEsMaxNodes] fp64 node rates a_k
  double* part;      // [B][T1][L][kEsMaxNodes] moments of each tile
  float* coef;       // [B][L][kEsMaxNodes] c_k (fp32 rows)
  double* coef64;    // [B][L][kEsMaxNodes] c_k (fp64 rows)
  int64_t T1;        // moments tiles per row
};

__host__ __device__ inline int64_t es_tiles(int64_t V, int tile) { return (V + tile - 1) / tile; }
__host__ __device__ inline int es_pad(int nk) { return (nk + kEsNB - 1) / kEsNB * kEsNB; }

__device__ __forceinline__ double wave_min64(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmin(v, __shfl_xor(v, off, 64));
  return v;
}
__device__ __forceinline__ double wave_max64(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off, 64));
  return v;
}

// ------------------------------------------------------------------ statistics
// grid (T1, B, L): min / max positive weight, count, zero-weight mass and bad
// values of law l = blockIdx.z over one tile of the row.
__global__ __launch_bounds__(kEsThreads) void es_stats_kernel(const float* __restrict__ p,
                                                               const float* __restrict__ q1,
                                                               const float* __restrict__ q2, int64_t V, EsWork es) {
  const int64_t t = blockIdx.x, b = blockIdx.y;
  const int l = blockIdx.z, L = gridDim.z;
  const float* pb = p + b * V;
  const float* qb = (l == 0 ? q1 : q2) + b * V;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  double wmin = INFINITY, wmax = 0.0;
  int npos = 0, bad = 0;
  double q0 = 0.0;
  const int64_t base = t * kEsMomTile;
#pragma unroll 4
  for (int i = 0; i < kEsMomPer; ++i) {
    const int64_t x = base + i * kEsThreads + tid;
    if (x >= V) break;
    const float pv = pb[x], qv = qb[x];
    bad |= (int)bad_prob(pv) | (int)bad_prob(qv);
    if (qv > 0.0f) {
      if (pv > 0.0f) {
        const double w = (double)pv / (double)qv;
        wmin = fmin(wmin, w);
        wmax = fmax(wmax, w);
        ++npos;
      } else {
        q0 += (double)qv;
      }
    }
  }
  wmin = wave_min64(wmin);
  wmax = wave_max64(wmax);
  npos = wave_sum_int(npos);
  bad = wave_sum_int(bad);
  q0 = wave_sum(q0);
  __shared__ EsTileStat s[kEsThreads / 64];
  if (lane == 0) {
    s[wid].wmin = wmin;
    s[wid].wmax = wmax;
    s[wid].npos = npos;
    s[wid].bad = bad;
    s[wid].q0 = q0;
  }
  __syncthreads();
  if (tid == 0) {
    EsTileStat o = s[0];
    for (int i = 1; i < kEsThreads / 64; ++i) {
      o.wmin = fmin(o.wmin, s[i].wmin);
      o.wmax = fmax(o.wmax, s[i].wmax);
      o.npos += s[i].npos;
      o.bad |= s[i].bad;
      o.q0 += s[i].q0;
    }
    es.stat[(b * es.T1 + t) * L + l] = o;
  }
}

// ------------------------------------------------------------------ plan
// One wave per row: the row's totals (tiles summed in a fixed order), its
// weight scale, node range and node table.  K >= 2 identical drafts (L = 1)
// or two draft laws (L = 2, K = 2).
__global__ __launch_bounds__(64) void es_plan_kernel(int K, int L, EsWork es,
                                                      int32_t* __restrict__ row_status) {
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  double wmin[2] = {INFINITY, INFINITY}, wmax[2] = {0.0, 0.0};
  int npos[2] = {0, 0}, bad = 0;
  double q0[2] = {0.0, 0.0};
  for (int64_t t = lane; t < es.T1; t += 64) {
    for (int l = 0; l < L; ++l) {
      const EsTileStat s = es.stat[(b * es.T1 + t) * L + l];
      wmin[l] = fmin(wmin[l], s.wmin);
      wmax[l] = fmax(wmax[l], s.wmax);
      npos[l] += s.npos;
      bad |= s.bad;
      q0[l] += s.q0;
    }
  }
  for (int l = 0; l < 2; ++l) {
    wmin[l] = wave_min64(wmin[l]);
    wmax[l] = wave_max64(wmax[l]);
    npos[l] = wave_sum_int(npos[l]);
    q0[l] = wave_sum(q0[l]);
  }
  bad = wave_sum_int(bad);
  EsPlan pl;
  pl.flags = bad ? kRowBadProb : 0;
  pl.k_lo = 0;
  pl.nk = 0;
  pl.sigma = 0;
  pl.wide = 0;
  pl.w64 = 0;
  pl.pad[0] = pl.pad[1] = 0;
  pl.q0[0] = q0[0];
  pl.q0[1] = q0[1];
  pl.pad2[0] = pl.pad2[1] = 0.0;
  const bool any = (L == 1) ? npos[0] > 0 : (npos[0] > 0 && npos[1] > 0);
  if (!pl.flags && any) {
    double lo = wmin[0], hi = wmax[0];
    if (L == 2) {
      lo = fmin(lo, wmin[1]);
      hi = fmax(hi, wmax[1]);
    }
    int e_lo, e_hi;
    frexp(lo, &e_lo);
    frexp(hi, &e_hi);
    pl.sigma = -((e_lo + e_hi) >> 1);
    pl.wide = (e_hi - e_lo) > kEsWideRange;
    pl.w64 = e_lo < -124 || e_hi > 126;  // an fp32 ratio p/q could be denormal or overflow
    // smallest and largest denominator of the row (scaled weights, fp64)
    double dmin, dmax;
    if (L == 1) {
      const double a = ldexp(wmin[0], pl.sigma), z = ldexp(wmax[0], pl.sigma);
      // K = 2 takes the zero-weight tokens in closed form; K >= 3 keeps them in S (denominator w(y) alone)
      dmin = (K == 2 || q0[0] == 0.0) ? K * a : a;
      dmax = K * z;
    } else {
      dmin = ldexp(wmin[0], pl.sigma) + ldexp(wmin[1], pl.sigma);
      dmax = ldexp(wmax[0], pl.sigma) + ldexp(wmax[1], pl.sigma);
    }
    const int k_lo = (int)floor((kEsLnEps - log(dmax)) / kEsStep);
    const int k_hi = (int)ceil((kEsLnLnInvEps - log(dmin)) / kEsStep);
    pl.k_lo = k_lo;
    pl.nk = k_hi - k_lo + 1;
    if (pl.nk > kEsMaxNodes) {  // only rows with probabilities far above 1 get here
      pl.flags = kRowRange;
      pl.nk = 0;
    }
  }
  if (lane == 0) {
    es.plan[b] = pl;
    if (row_status && pl.flags) row_status[b] |= pl.flags;
  }
  // node table, padded to whole blocks (padding rates are 1: their coefficients are 0)
  const int np = es_pad(pl.nk);
  for (int k = lane; k < np; k += 64) {
    const double a = (k < pl.nk) ? exp((double)(pl.k_lo + k) * kEsStep) : 1.0;
    es.alpha[b * kEsMaxNodes + k] = a;
    es.beta[b * kEsMaxNodes + k] = (float)(a * kEsLog2e);
  }
}

// Scaled weight w' = (p / q) 2^sigma in the row's precision.  fp32 rows take the
// correctly rounded fp32 ratio (equal to the fp64 ratio rounded once) unless a
// ratio of the row leaves the fp32 normal range.
template <typename Real>
__device__ __forceinline__ Real es_weight(float p, float q, const EsPlan& pl);
template <>
__device__ __forceinline__ float es_weight<float>(float p, float q, const EsPlan& pl) {
  return pl.w64 ? (float)ldexp((double)p / (double)q, pl.sigma) : ldexpf(p / q, pl.sigma);
}
template <>
__device__ __forceinline__ double es_weight<double>(float p, float q, const EsPlan& pl) {
  return ldexp((double)p / (double)q, pl.sigma);
}

__device__ __forceinline__ float es_fma(float a, float b, float c) { return fmaf(a, b, c); }
__device__ __forceinline__ double es_fma(double a, double b, double c) { return ::fma(a, b, c); }

// exp(-a w) from the node rate in the row's precision
__device__ __forceinline__ float es_decay(float beta, float w) { return __builtin_amdgcn_exp2f(-beta * w); }
__device__ __forceinline__ double es_decay(double alpha, double w) { return exp(-alpha * w); }

// The node tables are read-only inside the sweeps and uniform across a
// workgroup: reading them through the constant address space lets every wave
// take them with scalar loads into SGPRs.
template <typename T>
using const_as = const __attribute__((address_space(4))) T;

template <typename Real>
__device__ __forceinline__ const_as<Real>* es_rates(const EsWork& es, int64_t b);
template <>
__device__ __forceinline__ const_as<float>* es_rates<float>(const EsWork& es, int64_t b) {
  return (const_as<float>*)(es.beta + b * kEsMaxNodes);
}
template <>
__device__ __forceinline__ const_as<double>* es_rates<double>(const EsWork& es, int64_t b) {
  return (const_as<double>*)(es.alpha + b * kEsMaxNodes);
}

// Block-wide compaction: every thread holds `per` flags; returns this thread's
// first slot and (via total) the number of set flags in the block.
template <int per>
__device__ __forceinline__ int block_compact_offset(const bool (&flag)[per], int* s_wave, int& total) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int c = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) c += flag[i];
  const int incl = wave_inclusive_scan_int(c, lane);
  if (lane == 63) s_wave[wid] = incl;
  __syncthreads();
  int off = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < kEsThreads / 64; ++i) {
    off += (i < wid) ? s_wave[i] : 0;
    total += s_wave[i];
  }
  return off + incl - c;
}

// One halving stage of a wave reduce-scatter: lanes with bit OFF set keep the
// upper HALF of their values, the others the lower HALF; each kept value gets
// its partner lane's copy added.
template <int OFF, int HALF, typename Real>
__device__ __forceinline__ void rs_stage(Real (&v)[16], int lane) {
  const bool up = (lane & OFF) != 0;
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const Real send = up ? v[i] : v[i + HALF];
    const Real keep = up ? v[i + HALF] : v[i];
    v[i] = keep + __shfl_xor(send, OFF, 64);
  }
}

// Sum of 16 per-lane values over the 64 lanes of a wave, scattered: afterwards
// lane l holds the total of value (l >> 2) (fixed order, deterministic).
template <typename Real>
__device__ __forceinline__ Real wave_reduce_scatter16(Real (&v)[16], int lane) {
  rs_stage<32, 8>(v, lane);
  rs_stage<16, 4>(v, lane);
  rs_stage<8, 2>(v, lane);
  rs_stage<4, 1>(v, lane);
  Real x = v[0];
  x += __shfl_xor(x, 2, 64);
  x += __shfl_xor(x, 1, 64);
  return x;
}

// ------------------------------------------------------------------ moments
// grid (T1, B, L): S_k over one tile of law l: sum of q(x) exp(-a_k w'(x)) over
// its positive-weight tokens, for every node of the row.  Tokens are compacted
// into LDS; each thread keeps 16 node sums for its tokens, which are summed
// over the wave (reduce-scatter) and then over the four waves.
template <typename Real>
__global__ __launch_bounds__(kEsThreads) void es_moments_kernel(const float* __restrict__ p,
                                                                 const float* __restrict__ q1,
                                                                 const float* __restrict__ q2, int64_t V,
                                                                 EsWork es) {
  const int64_t t = blockIdx.x, b = blockIdx.y;
  const int l = blockIdx.z, L = gridDim.z;
  const EsPlan pl = es.plan[b];
  if (pl.flags || pl.nk == 0 || pl.wide != (sizeof(Real) == 8)) return;
  const float* pb = p + b * V;
  const float* qb = (l == 0 ? q1 : q2) + b * V;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  __shared__ Real s_w[kEsMomTile];
  __shared__ float s_q[kEsMomTile];
  __shared__ Real s_red[kEsThreads / 64][kEsMaxNodes];
  __shared__ int s_wave[kEsThreads / 64];

  const int64_t base = t * kEsMomTile;
  bool pos[kEsMomPer];
  Real wv[kEsMomPer];
  float qv[kEsMomPer];
#pragma unroll
  for (int i = 0; i < kEsMomPer; ++i) {
    const int64_t x = base + i * kEsThreads + tid;
    const float pp = (x < V) ? pb[x] : 0.0f;
    const float qq = (x < V) ? qb[x] : 0.0f;
    pos[i] = pp > 0.0f && qq > 0.0f;
    wv[i] = pos[i] ? es_weight<Real>(pp, qq, pl) : (Real)0;
    qv[i] = qq;
  }
  int n = 0;
  int off = block_compact_offset<kEsMomPer>(pos, s_wave, n);
#pragma unroll
  for (int i = 0; i < kEsMomPer; ++i) {
    if (pos[i]) {
      s_w[off] = wv[i];
      s_q[off] = qv[i];
      ++off;
    }
  }
  __syncthreads();
  const int M = (n + kEsThreads - 1) / kEsThreads;
  const_as<Real>* rate = es_rates<Real>(es, b);
  const int np = es_pad(pl.nk);
  for (int nb = 0; nb < np; nb += kEsNB) {
    Real rt[kEsNB], acc[kEsNB];
#pragma unroll
    for (int i = 0; i < kEsNB; ++i) {
      rt[i] = rate[nb + i];
      acc[i] = (Real)0;
    }
    for (int m = 0; m < M; ++m) {
      const int j = tid + m * kEsThreads;
      const Real w = (j < n) ? s_w[j] : (Real)0;
      const Real qq = (j < n) ? (Real)s_q[j] : (Real)0;
#pragma unroll
      for (int i = 0; i < kEsNB; ++i) acc[i] = es_fma(qq, es_decay(rt[i], w), acc[i]);
    }
    const Real tot = wave_reduce_scatter16<Real>(acc, lane);
    if ((lane & 3) == 0) s_red[wid][nb + (lane >> 2)] = tot;
  }
  __syncthreads();
  double* out = es.part + ((b * es.T1 + t) * L + l) * kEsMaxNodes;
  for (int k = tid; k < pl.nk; k += kEsThreads) {
    Real s = s_red[0][k];
#pragma unroll
    for (int i = 1; i < kEsThreads / 64; ++i) s += s_red[i][k];
    out[k] = (double)s;
  }
}


// ------------------------------------------------------------------ coefficients
// One workgroup per row: the moments of all tiles summed in tile order (fp64)
// and the node coefficients.  K i.i.d. drafts: c_k = K h a_k S_k^(K-1) (K >= 3
// keeps the zero-weight mass Q0 in S).  Two laws: the queries of law 1 take
// h a_k S_k of law 2 and the queries of law 2 take h a_k S_k of law 1.
__global__ __launch_bounds__(kEsThreads) void es_coef_kernel(int K, int L, EsWork es) {
  const int64_t b = blockIdx.x;
  const EsPlan pl = es.plan[b];
  if (pl.flags || pl.nk == 0) return;
  const int np = es_pad(pl.nk);
  for (int k = threadIdx.x; k < np; k += kEsThreads) {
    double S[2] = {0.0, 0.0};
    if (k < pl.nk) {
      for (int64_t t = 0; t < es.T1; ++t)
        for (int l = 0; l < L; ++l) S[l] += es.part[((b * es.T1 + t) * L + l) * kEsMaxNodes + k];
    }
    const double ha = kEsStep * es.alpha[b * kEsMaxNodes + k];
    double c[2];
    if (L == 1) {
      const double s = S[0] + (K >= 3 ? pl.q0[0] : 0.0);
      double sp = 1.0;
      for (int j = 1; j < K; ++j) sp *= s;
      c[0] = (double)K * ha * sp;
    } else {
      c[0] = ha * S[1];
      c[1] = ha * S[0];
    }
    for (int l = 0; l < L; ++l) {
      const double v = (k < pl.nk) ? c[l] : 0.0;
      es.coef[(b * L + l) * kEsMaxNodes + k] = (float)v;
      es.coef64[(b * L + l) * kEsMaxNodes + k] = v;
    }
  }
}

template <typename Real>
__device__ __forceinline__ const_as<Real>* es_coefs(const EsWork& es, int64_t b, int l, int L);
template <>
__device__ __forceinline__ const_as<float>* es_coefs<float>(const EsWork& es, int64_t b, int l, int L) {
  return (const_as<float>*)(es.coef + (b * L + l) * kEsMaxNodes);
}
template <>
__device__ __forceinline__ const_as<double>* es_coefs<double>(const EsWork& es, int64_t b, int l, int L) {
  return (const_as<double>*)(es.coef64 + (b * L + l) * kEsMaxNodes);
}

// ------------------------------------------------------------------ evaluation
// grid (T2, B): r over one tile of 2048 tokens.  The positive-weight tokens of
// each law are compacted into LDS; a thread evaluates four of them at a time
// over all nodes (sum_k c_k exp(-a_k w'(y)), fp32 blocks of 16 nodes folded
// into the running sum), and r is assembled per token with the zero-weight
// closed forms.  The fp32 instantiation also writes flagged rows (NaN) and rows
// without a quadrature term.
template <typename Real, int L>
__global__ __launch_bounds__(kEsThreads) void es_eval_kernel(const float* __restrict__ p,
                                                              const float* __restrict__ q1,
                                                              const float* __restrict__ q2, int64_t V, int K,
                                                              float* __restrict__ r, EsWork es) {
  const int64_t t = blockIdx.x, b = blockIdx.y;
  const EsPlan pl = es.plan[b];
  if (pl.wide != (sizeof(Real) == 8)) return;
  const float* pb = p + b * V;
  float* rb = r + b * V;
  const int tid = threadIdx.x;
  const int64_t base = t * kEsEvalTile;
  if (pl.flags) {
#pragma unroll
    for (int i = 0; i < kEsEvalPer; ++i) {
      const int64_t x = base + i * kEsThreads + tid;
      if (x < V) rb[x] = NAN;
    }
    return;
  }
  __shared__ Real s_w[kEsEvalTile];
  __shared__ int s_pos[kEsEvalTile];
  __shared__ Real s_acc[kEsEvalTile];
  __shared__ int s_wave[kEsThreads / 64];
  float pv[kEsEvalPer], qv[L][kEsEvalPer];
#pragma unroll
  for (int i = 0; i < kEsEvalPer; ++i) {
    const int64_t x = base + i * kEsThreads + tid;
    pv[i] = (x < V) ? pb[x] : 0.0f;
    qv[0][i] = (x < V) ? q1[b * V + x] : 0.0f;
    if (L == 2) qv[L - 1][i] = (x < V) ? q2[b * V + x] : 0.0f;
    s_acc[i * kEsThreads + tid] = (Real)0;
  }
  if (pl.nk > 0) {
    const_as<Real>* rate = es_rates<Real>(es, b);
    const int np = es_pad(pl.nk);
#pragma unroll
    for (int l = 0; l < L; ++l) {
      bool pos[kEsEvalPer];
#pragma unroll
      for (int i = 0; i < kEsEvalPer; ++i) pos[i] = pv[i] > 0.0f && qv[l][i] > 0.0f;
      int n = 0;
      int off = block_compact_offset<kEsEvalPer>(pos, s_wave, n);
#pragma unroll
      for (int i = 0; i < kEsEvalPer; ++i) {
        if (pos[i]) {
          s_w[off] = es_weight<Real>(pv[i], qv[l][i], pl);
          s_pos[off] = i * kEsThreads + tid;
          ++off;
        }
      }
      __syncthreads();
      const_as<Real>* cf = es_coefs<Real>(es, b, l, L);
      for (int j0 = 0; j0 < n; j0 += 4 * kEsThreads) {
        Real w[4], acc[4];
        int ps[4];
        bool ok[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = j0 + e * kEsThreads + tid;
          ok[e] = j < n;
          w[e] = ok[e] ? s_w[j] : (Real)0;
          ps[e] = ok[e] ? s_pos[j] : 0;
          acc[e] = (Real)0;
        }
        for (int nb = 0; nb < np; nb += kEsNB) {
          Real blk[4] = {(Real)0, (Real)0, (Real)0, (Real)0};
#pragma unroll
          for (int i = 0; i < kEsNB; ++i) {
            const Real rt = rate[nb + i], c = cf[nb + i];
#pragma unroll
            for (int e = 0; e < 4; ++e) blk[e] = es_fma(c, es_decay(rt, w[e]), blk[e]);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += blk[e];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (ok[e]) s_acc[ps[e]] += acc[e];  // one entry per token and law: no two threads share a slot
      }
      __syncthreads();  // s_w / s_pos are rebuilt for the next law; s_acc is read below
    }
  }
  const double q0a = pl.q0[0], q0b = (L == 2) ? pl.q0[1] : 0.0;
  double zw = q0a;  // K i.i.d. drafts: Q0^(K-1)
  for (int j = 2; j < K; ++j) zw *= q0a;
#pragma unroll
  for (int i = 0; i < kEsEvalPer; ++i) {
    const int64_t x = base + i * kEsThreads + tid;
    if (x >= V) break;
    const double pp = (double)pv[i];
    const double quad = ldexp((double)s_acc[i * kEsThreads + tid], pl.sigma);
    double v = 0.0;
    if (L == 1) {
      const double qq = (double)qv[0][i];
      if (qq > 0.0) v = (pp > 0.0) ? pp * quad + (K == 2 ? 2.0 * qq * q0a : 0.0) : qq * zw;
    } else {
      // two laws: a zero-weight pole of the other draft adds q_i(y) Qj_0; a zero target splits it in half
      const double a = (double)qv[0][i], c = (double)qv[L - 1][i];
      if (pp > 0.0) {
        v = pp * quad + (a > 0.0 ? a * q0b : 0.0) + (c > 0.0 ? c * q0a : 0.0);
      } else {
        v = 0.5 * ((a > 0.0 ? a * q0b : 0.0) + (c > 0.0 ? c * q0a : 0.0));
      }
    }
    rb[x] = (float)v;
  }
}

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

void carve_es(void* base, int64_t B, int64_t V, int L, EsWork* es) {
  const int64_t T1 = es_tiles(V, kEsMomTile);
  char* c = static_cast<char*>(base);
  es->stat = reinterpret_cast<EsTileStat*>(c);
  c += align256(sizeof(EsTileStat) * B * T1 * L);
  es->plan = reinterpret_cast<EsPlan*>(c);
  c += align256(sizeof(EsPlan) * B);
  es->beta = reinterpret_cast<float*>(c);
  c += align256(sizeof(float) * B * kEsMaxNodes);
  es->alpha = reinterpret_cast<double*>(c);
  c += align256(sizeof(double) * B * kEsMaxNodes);
  es->part = reinterpret_cast<double*>(c);
  c += align256(sizeof(double) * B * T1 * L * kEsMaxNodes);
  es->coef = reinterpret_cast<float*>(c);
  c += align256(sizeof(float) * B * L * kEsMaxNodes);
  es->coef64 = reinterpret_cast<double*>(c);
  es->T1 = T1;
}

}  // namespace

size_t workspace_bytes_expsum(int64_t B, int64_t V, int L) {
  const int64_t T1 = es_tiles(V, kEsMomTile);
  return align256(sizeof(EsTileStat) * B * T1 * L) + align256(sizeof(EsPlan) * B) +
         align256(sizeof(float) * B * kEsMaxNodes) + align256(sizeof(double) * B * kEsMaxNodes) +
         align256(sizeof(double) * B * T1 * L * kEsMaxNodes) + align256(sizeof(float) * B * L * kEsMaxNodes) +
         align256(sizeof(double) * B * L * kEsMaxNodes);
}

// q2 == nullptr: K i.i.d. drafts from q1; else two draft laws (K = 2).
hipError_t launch_induced_expsum(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, int K,
                                 float* r, int32_t* row_status, void* workspace, hipStream_t st) {
  const int L = (q2 != nullptr) ? 2 : 1;
  EsWork es;
  carve_es(workspace, B, V, L, &es);
  const int64_t T2 = es_tiles(V, kEsEvalTile);
  const dim3 g1((unsigned)es.T1, (unsigned)B, (unsigned)L);
  hipLaunchKernelGGL(es_stats_kernel, g1, dim3(kEsThreads), 0, st, p, q1, q2, V, es);
  hipLaunchKernelGGL(es_plan_kernel, dim3((unsigned)B), dim3(64), 0, st, K, L, es, row_status);
  hipLaunchKernelGGL(es_moments_kernel<float>, g1, dim3(kEsThreads), 0, st, p, q1, q2, V, es);
  hipLaunchKernelGGL(es_moments_kernel<double>, g1, dim3(kEsThreads), 0, st, p, q1, q2, V, es);
  hipLaunchKernelGGL(es_coef_kernel, dim3((unsigned)B), dim3(kEsThreads), 0, st, K, L, es);
  const dim3 g2((unsigned)T2, (unsigned)B);
  if (L == 1) {
    hipLaunchKernelGGL((es_eval_kernel<float, 1>), g2, dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, es);
    hipLaunchKernelGGL((es_eval_kernel<double, 1>), g2, dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, es);
  } else {
    hipLaunchKernelGGL((es_eval_kernel<float, 2>), g2, dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, es);
    hipLaunchKernelGGL((es_eval_kernel<double, 2>), g2, dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, es);
  }
  return hipGetLastError();
}

// Successive pairwise reduction (Remark 4) with every stage law by the quadrature.
hipError_t launch_induced_successive_expsum(const float* p, const float* q, int64_t B, int64_t V, int K,
                                            float* r_stages, int32_t* row_status, void* workspace, hipStream_t st) {
  hipError_t e = launch_induced_expsum(p, q, nullptr, B, V, 2, r_stages, row_status, workspace, st);
  const int64_t plane = B * V;
  for (int j = 1; j < K - 1 && e == hipSuccess; ++j)
    e = launch_induced_expsum(p, r_stages + (j - 1) * plane, q, B, V, 2, r_stages + j * plane, row_status,
                              workspace, st);
  return e;
}

}  // namespace mdss
