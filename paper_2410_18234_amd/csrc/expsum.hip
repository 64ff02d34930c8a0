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
// t_k = k h (k an integer, the same grid for every row) turns the O(n^K) sum
// into O(n) work per node:
//   moments    S_k = sum_x q(x) exp(-a_k w(x)),   a_k = e^(t_k),
//   evaluation r(y) = p(y) sum_k c_k exp(-a_k w(y)),  c_k = K h a_k S_k^(K-1).
// Error of the rule (relative, for every D, independently of D): by Poisson
// summation the integrand exp(t - D e^t) has Fourier transform
// D^(-1+iv) Gamma(1 - iv), so the step-h sum differs from 1/D by at most
// 2 sum_{m>=1} |Gamma(1 + 2 pi i m / h)| / D, 4.8e-8 for h = 1/2.  A row's grid
// is cut where the left tail (t < t_lo: relative D e^t_lo) and the right tail
// (t > t_hi: relative exp(-D e^t_hi)) are below 1e-8 for every denominator of
// the row.  Every term is positive, so these relative bounds hold for the
// sums and for r; fp32 evaluation adds a few 1e-8.
//
// Windows.  Nodes where a_k w <= 1/4 for every token of a group are taken by an
// eight-term expansion of exp(-a_k w) in powers of a_k w (truncation below
// 4e-10 relative); nodes where a_k w > Z = 22 for a token drop that token's term.
// The drop is a truncation of the integral: a token x with weight w_x inside a
// denominator D >= w_x loses at most the part of its pair (or tuple) integral
// over a > Z / w_x, which relative to 1/D is at most e^(-Z D / w_x) (1 + h Z D / w_x)
// <= e^(-Z) (1 + h Z) = 3.3e-9 on the grid (the integrand is decreasing there),
// once on the moment side and once on the query side.  So a token needs
// exponentials only on the nodes with a_k w in (1/4, 22]: nine of them.  The
// evaluation gives every query token exactly those nine (its expansion of the
// grid below comes from a prefix table), as one polynomial of degree 10 in its
// a_k0 w per node row (interpolation error at most 4.7e-9 relative, so the
// budget is 8.1e-8 in all); the moments, a sum over tokens per
// node, give each run of 512 tokens of nearby weights (after a per-thread sort)
// the union of its tokens' windows.  Moments need no row-wide information, so
// they run first; one workgroup per row then merges the tiles, fixes the row's
// grid range, coefficients and prefix table; evaluation follows.
//
// Precision: each tile scales its weights by a power of two (w' = w 2^tau, the
// node rates by 2^-tau) and evaluates in fp32; a tile whose weight ratios leave
// the fp32 normal range or span more than 2^160 is redone in fp64 by the
// coefficient kernel, which then evaluates that row in fp64 as well.
// Zero-weight tokens (p = 0 < q) enter in closed form; a flagged row gets NaN.
#include "common.h"
#include "draw.h"
#include "expsum_poly.h"
#include "mdss.h"

#include <float.h>
#include <math.h>

#include <algorithm>
#include <mutex>

namespace mdss {

namespace {

constexpr int kEsThreads = 256;
constexpr int kEsWaves = kEsThreads / 64;
constexpr int kEsMomPer = 16;                           // tokens per thread, moments
constexpr int kEsMomTile = kEsThreads * kEsMomPer;      // 4096 tokens per moments tile
constexpr int kEsEvalPer = 8;                           // tokens per thread, evaluation
constexpr int kEsEvalTile = kEsThreads * kEsEvalPer;    // 2048 tokens per evaluation tile
constexpr int kEsMaxNodes = 480;                        // nodes of a row (weights spanning <= 2^300)
constexpr int kEsMaxWin = 496;                          // nodes of a tile window; table stride
constexpr int kEsTaylor = 8;                            // terms of the far-node expansion (j = 0..7)
constexpr int kEsPart = kEsTaylor + kEsMaxWin;          // per tile: power sums, then the window moments
constexpr double kEsStep = 0.5;                         // h
constexpr double kEsLnEps = -18.420680743952367;        // ln 1e-8: left-tail cut
constexpr double kEsLnLnInvEps = 2.9134941423228814;    // ln ln 1e8: right-tail cut
constexpr double kEsLnFar = -1.3862943611198906;        // ln 1/4: at or below, a node is taken by the expansion
constexpr double kEsLnZero = 3.0910424533583156;        // ln 22: above, a token's term is dropped
constexpr double kEsLog2e = 1.4426950408889634;
constexpr int kEsWideRange = 160;  // binary exponent range of a tile's weights kept in fp32
constexpr int kEsAtabRows = kEsMaxNodes + 16;  // polynomial rows of a row and law (bound of EsPlan::nrow)
constexpr int kEsTokNodesC = 9;                // node terms of a query token (a_k w in (1/4, 22.5])

// Per (row, moments tile, law).
struct alignas(64) EsTile {
  double wmin;   // smallest positive weight (+inf if none)
  double wmax;   // largest weight (0 if none)
  double pad0;
  double q0;     // draft mass of zero-weight tokens (q > 0 = p)
  int32_t npos;  // positive-weight tokens
  int32_t bad;   // a NaN, negative or infinite probability was read
  int32_t kt;    // last node taken by the expansion; the window is kt + 1 .. kt + nw
  int32_t nw;    // window length (0: no positive weight)
  int32_t wide;  // 1: the moments are taken in fp64 (by the coefficient kernel)
  int32_t small; // 1: a positive-weight token has a draft probability below the fp32 normal range
  int32_t pad[2];
};

// Per row.
struct alignas(64) EsPlan {
  int32_t flags;  // row status bits; a flagged row gets r = NaN
  int32_t k_lo;   // first node of the row's grid
  int32_t nk;     // nodes of the row's grid (0: no quadrature term)
  int32_t fp64;   // 1: the row is evaluated in fp64 by the coefficient kernel
  double q0[2];   // per law: draft mass of zero-weight tokens
  int32_t nrow;   // polynomial rows written per law: node rows 0 .. nrow - 1 (k0 = k_lo + i)
  int32_t pad_i;
  double pad[4];
};

struct EsWork {
  EsTile* tile;     // [B][T1][L]
  double* part;     // [B][T1][L][kEsPart] per tile: power sums T_j, then the moments of its window
  EsPlan* plan;     // [B]
  double* ptab;     // [B][L][kEsMaxNodes][kEsTaylor] B_j(k_lo + i) / j!: the expansion of the grid up to a node
  double* atab;     // [B][L][kEsAtabRows][kEsPolyLen] per-token polynomial of node row i (k0 = k_lo + i)
  int64_t T1, T2, T3;  // moments tiles, fp64 evaluation tiles, fp32 evaluation tiles (per row)
};

__host__ __device__ inline int64_t es_tiles(int64_t V, int tile) { return (V + tile - 1) / tile; }

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

__device__ __forceinline__ double es_wave_min(double v) { return wave_min64(v); }
__device__ __forceinline__ double es_wave_max(double v) { return wave_max64(v); }

// Nodes of a group whose positive weights lie in [wlo, whi]: up to kt, a_k whi
// <= 1/4 and the expansion takes them; after kt + nw, a_k wlo > 22 and every
// token's term is dropped; the window in between is summed with exponentials.
__device__ inline void es_window(double wlo, double whi, int& kt, int& nw) {
  kt = (int)floor((kEsLnFar - log(whi)) / kEsStep);
  const int z = (int)floor((kEsLnZero - log(wlo)) / kEsStep);
  nw = max(0, min(z - kt, kEsMaxWin));
}

// The same in fp32 for weights in the fp32 range (hardware log2; a boundary
// node off by one rounding of the logarithm keeps both bounds within 1e-5 of
// their limits, where exp(-z) is 1 or 0 to far below the rule's error).
__device__ inline void es_window_f32(float wlo, float whi, int& kt, int& nw) {
  constexpr float kLn2 = 0.69314718f;
  kt = (int)floorf(((float)kEsLnFar - __builtin_amdgcn_logf(whi) * kLn2) * (float)(1.0 / kEsStep));
  const int z = (int)floorf(((float)kEsLnZero - __builtin_amdgcn_logf(wlo) * kLn2) * (float)(1.0 / kEsStep));
  nw = max(0, min(z - kt, kEsMaxWin));
}
__device__ inline void es_scale_f32(float wlo, float whi, int& tau, int& range) {
  int e_lo, e_hi;
  frexpf(wlo, &e_lo);
  frexpf(whi, &e_hi);
  tau = -((e_lo + e_hi) >> 1);
  range = e_hi - e_lo;
}

// 1 / j! for the expansion exp(-u) = sum_j (-u)^j / j!
__device__ __forceinline__ double es_inv_fact(int j) {
  double f = 1.0;
  for (int i = 2; i <= j; ++i) f *= (double)i;
  return 1.0 / f;
}

// Power-of-two scale that centres [wlo, whi] on 1 and the binary range it spans.
__device__ inline void es_scale(double wlo, double whi, int& tau, int& range) {
  int e_lo, e_hi;
  frexp(wlo, &e_lo);
  frexp(whi, &e_hi);
  tau = -((e_lo + e_hi) >> 1);
  range = e_hi - e_lo;
}

// node rate of an fp64 tile: a_k 2^-tau
template <typename Real>
__device__ __forceinline__ Real es_rate(int k, int tau);
template <>
__device__ __forceinline__ double es_rate<double>(int k, int tau) {
  return ldexp(exp((double)k * kEsStep), -tau);
}

__device__ __forceinline__ float es_decay(float beta, float w) { return __builtin_amdgcn_exp2f(-beta * w); }
__device__ __forceinline__ double es_decay(double alpha, double w) { return exp(-alpha * w); }
__device__ __forceinline__ double es_fma(double a, double b, double c) { return ::fma(a, b, c); }

template <typename Real>
__device__ __forceinline__ Real es_ratio(float p, float q);
template <>
__device__ __forceinline__ float es_ratio<float>(float p, float q) {
  // reciprocal and product: within 2 ulp of p / q, the same value in every kernel
  return p * __builtin_amdgcn_rcpf(q);
}
// The same ratio for a draft probability below the fp32 normal range, whose
// reciprocal would overflow: q is scaled up by 2^64 first (p / q itself is
// often far inside the range: a draft at a low temperature puts its tail there).
// The kernels take it only in waves that hold such a q (a uniform branch).
__device__ __forceinline__ float es_ratio_small_q(float p, float q) {
  return (p * __builtin_amdgcn_rcpf(q * 0x1p64f)) * 0x1p64f;
}
// positive fp32 denormal (class bit 7; bits 0-9: signalling NaN, quiet NaN, -inf, -normal,
// -denormal, -0, +0, +denormal, +normal, +inf)
__device__ __forceinline__ bool es_denormal(float q) { return __builtin_amdgcn_classf(q, 0x80); }
template <>
__device__ __forceinline__ double es_ratio<double>(float p, float q) {
  return (double)p / (double)q;
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
  for (int i = 0; i < kEsWaves; ++i) {
    off += (i < wid) ? s_wave[i] : 0;
    total += s_wave[i];
  }
  return off + incl - c;
}

// One halving stage of a wave reduce-scatter: lanes with bit OFF set keep the
// upper HALF of their values, the others the lower HALF; each kept value gets
// its partner lane's copy added.
template <int OFF, int HALF, int N, typename Real>
__device__ __forceinline__ void rs_stage(Real (&v)[N], int lane) {
  const bool up = (lane & OFF) != 0;
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const Real send = up ? v[i] : v[i + HALF];
    const Real keep = up ? v[i + HALF] : v[i];
    v[i] = keep + __shfl_xor(send, OFF, 64);
  }
}

// Sum of NB per-lane values over the 64 lanes of a wave, scattered: afterwards
// lane l holds the total of value l / (64 / NB) (fixed order, deterministic).
template <int NB, typename Real>
__device__ __forceinline__ Real wave_reduce_scatter(Real (&v)[NB], int lane) {
  static_assert(NB == 4 || NB == 8 || NB == 16, "block sizes");
  rs_stage<32, NB / 2>(v, lane);
  rs_stage<16, NB / 4>(v, lane);
  if constexpr (NB >= 8) rs_stage<8, NB / 8>(v, lane);
  if constexpr (NB >= 16) rs_stage<4, NB / 16>(v, lane);
  Real x = v[0];
#pragma unroll
  for (int off = 64 / NB / 2; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// fp32: the same sums without LDS traffic.  Values are split by lane bit 2 and
// bit 3 within 16-lane rows through DPP rotations (a rotation by 4 or 8 always
// flips that bit and keeps the others below bit 4, so every lane is paired
// once), by bits 4 and 5 through the row and half swaps of gfx950; the bits
// left over are summed (swaps with the value itself, quad permutations).  For
// NB = 16 / 8 / 4 / 2 / 1 lane l ends with the total of value 8 b2 + 4 b3 + 2 b4
// + b5 / 4 b2 + 2 b3 + b4 / 2 b2 + b3 / b2 / 0 (b_i = bit i of l);
// es_scatter_node and es_scatter_writer name that value and one lane holding it.
template <int HALF, int N, int CTRL>
__device__ __forceinline__ void rs_dpp(float (&v)[N], bool up) {
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const float send = up ? v[i] : v[i + HALF];
    const float keep = up ? v[i + HALF] : v[i];
    v[i] = keep + dpp<CTRL>(send);
  }
}
template <int HALF, int N, bool ROW>
__device__ __forceinline__ void rs_swap(float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < HALF; ++i) {
    const auto r = ROW ? __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]), __float_as_uint(v[i + HALF]), false, false)
                       : __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]), __float_as_uint(v[i + HALF]), false, false);
    v[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
}
template <bool ROW>
__device__ __forceinline__ float sum_swap(float x) {
  const auto r = ROW ? __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false)
                     : __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
template <int NB>
__device__ __forceinline__ float wave_reduce_scatter_f32(float (&v)[NB], int lane) {
  static_assert(NB == 1 || NB == 2 || NB == 4 || NB == 8 || NB == 16, "block sizes");
  float x;
  if constexpr (NB <= 2) {
    if constexpr (NB == 2) {
      rs_dpp<1, NB, 0x124>(v, (lane & 4) != 0);  // row_ror:4
      x = v[0];
    } else {
      x = v[0];
      x += dpp<0x124>(x);
    }
    x += dpp<0x128>(x);  // row_ror:8
    x = sum_swap<false>(sum_swap<true>(x));
    x += dpp<0xB1>(x);
    x += dpp<0x4E>(x);
    return x;
  }
  rs_dpp<NB / 2, NB, 0x124>(v, (lane & 4) != 0);  // row_ror:4
  rs_dpp<NB / 4, NB, 0x128>(v, (lane & 8) != 0);  // row_ror:8
  if constexpr (NB == 16) {
    rs_swap<2, NB, true>(v);
    rs_swap<1, NB, false>(v);
    x = v[0];
  } else if constexpr (NB == 8) {
    rs_swap<1, NB, true>(v);
    x = sum_swap<false>(v[0]);
  } else {
    x = sum_swap<false>(sum_swap<true>(v[0]));
  }
  x += dpp<0xB1>(x);  // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);  // quad_perm [2,3,0,1]
  return x;
}
template <int NB>
__device__ __forceinline__ int es_scatter_node(int lane) {
  const int b2 = (lane >> 2) & 1, b3 = (lane >> 3) & 1, b4 = (lane >> 4) & 1, b5 = (lane >> 5) & 1;
  return NB == 16 ? 8 * b2 + 4 * b3 + 2 * b4 + b5
                  : (NB == 8 ? 4 * b2 + 2 * b3 + b4 : (NB == 4 ? 2 * b2 + b3 : (NB == 2 ? b2 : 0)));
}
template <int NB>
__device__ __forceinline__ bool es_scatter_writer(int lane) {
  return NB == 16 ? (lane & 3) == 0
                  : (NB == 8 ? (lane & 0x23) == 0
                             : (NB == 4 ? (lane & 0x33) == 0 : (NB == 2 ? (lane & 0x3B) == 0 : lane == 0)));
}

// Minimum / maximum of a float over the 64 lanes of a wave, in every lane
// (quad permutations, row rotations by 4 and 8, then the gfx950 row and half
// swaps; all lanes must be active).
template <bool MAX>
__device__ __forceinline__ float es_pick(float a, float b) {
  return MAX ? fmaxf(a, b) : fminf(a, b);
}
template <bool MAX>
__device__ __forceinline__ float es_wave_ext(float x) {
  x = es_pick<MAX>(x, dpp<0xB1>(x));   // quad_perm [1,0,3,2]
  x = es_pick<MAX>(x, dpp<0x4E>(x));   // quad_perm [2,3,0,1]
  x = es_pick<MAX>(x, dpp<0x124>(x));  // row_ror:4
  x = es_pick<MAX>(x, dpp<0x128>(x));  // row_ror:8
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = es_pick<MAX>(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return es_pick<MAX>(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// The same for the bit patterns of non-negative floats (+0 .. +inf order as unsigned
// integers): no NaN handling around each step, and each step one DPP-fused min / max.
template <bool MAX>
__device__ __forceinline__ uint32_t es_pick_u(uint32_t a, uint32_t b) {
  return MAX ? (a > b ? a : b) : (a < b ? a : b);
}
template <bool MAX>
__device__ __forceinline__ uint32_t es_wave_ext_u(uint32_t x) {
  x = es_pick_u<MAX>(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
  x = es_pick_u<MAX>(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
  x = es_pick_u<MAX>(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x124, 0xF, 0xF, false));  // row_ror:4
  x = es_pick_u<MAX>(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x128, 0xF, 0xF, false));  // row_ror:8
  auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = es_pick_u<MAX>(r[0], r[1]);
  r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return es_pick_u<MAX>(r[0], r[1]);
}
// the same, made explicit as a wave-uniform value
__device__ __forceinline__ float es_uniform_min(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(es_wave_ext<false>(x))));
}
__device__ __forceinline__ float es_uniform_max(float x) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(es_wave_ext<true>(x))));
}

// ------------------------------------------------------------------ moments
// The fp64 path: statistics and moments of one tile of one law that the fp32
// kernel left aside (a ratio outside the fp32 normal range or a weight span above
// 2^160), taken by the coefficient kernel; the same record layout, tile windows
// on a compacted token list (no sort).
template <int NB, typename Real>
__device__ __forceinline__ void es_moments_block(const Real* __restrict__ s_w, const float* __restrict__ s_q,
                                                 const Real* __restrict__ s_rate, int M, int nb, int tid, int lane,
                                                 int wid, Real (*s_red)[kEsMaxWin]) {
  Real rt[NB], acc[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    rt[i] = s_rate[nb + i];
    acc[i] = (Real)0;
  }
  for (int m = 0; m < M; ++m) {
    const int j = tid + m * kEsThreads;
    const Real w = s_w[j];
    const Real qq = (Real)s_q[j];
#pragma unroll
    for (int i = 0; i < NB; ++i) acc[i] = es_fma(qq, es_decay(rt[i], w), acc[i]);
  }
  const Real tot = wave_reduce_scatter<NB, Real>(acc, lane);
  if ((lane & (64 / NB - 1)) == 0) s_red[wid][nb + lane / (64 / NB)] = tot;
}

template <typename Real>
__device__ void es_moments_tile(const float* __restrict__ pb, const float* __restrict__ qb, int64_t V, int64_t t,
                                EsTile* __restrict__ rec, double* __restrict__ part) {
  static_assert(sizeof(Real) == 8, "the fp64 path");
  __shared__ Real s_w[kEsMomTile];
  __shared__ float s_q[kEsMomTile];
  __shared__ Real s_red[kEsWaves][kEsMaxWin];
  __shared__ Real s_rate[kEsMaxWin];
  __shared__ Real s_tay[kEsWaves][kEsTaylor];
  __shared__ int s_wave[kEsWaves];
  __shared__ double s_d[kEsWaves][4];
  __shared__ int s_i[kEsWaves][2];
  __shared__ int s_dec[4];  // ka, nw, tau, proceed
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t base = t * kEsMomTile;

  bool pos[kEsMomPer];
  Real wv[kEsMomPer];
  float qv[kEsMomPer];
  Real wlo = (Real)INFINITY, whi = (Real)0;
  float q0f = 0.0f;
  int npos = 0, bad = 0;
#pragma unroll
  for (int i = 0; i < kEsMomPer; ++i) {
    const int64_t x = base + i * kEsThreads + tid;
    const float pp = (x < V) ? pb[x] : 0.0f;
    const float qq = (x < V) ? qb[x] : 0.0f;
    bad |= (int)bad_prob(pp) | (int)bad_prob(qq);
    pos[i] = pp > 0.0f && qq > 0.0f;
    const Real w = pos[i] ? es_ratio<Real>(pp, qq) : (Real)0;
    wv[i] = w;
    qv[i] = qq;
    wlo = pos[i] ? fmin(wlo, w) : wlo;
    whi = pos[i] ? fmax(whi, w) : whi;
    npos += pos[i];
    q0f += (qq > 0.0f && pp == 0.0f) ? qq : 0.0f;
  }
  const double wmin_w = (double)es_wave_min(wlo), wmax_w = (double)es_wave_max(whi);
  const double q0 = wave_sum((double)q0f);
  npos = wave_sum_int(npos);
  bad = wave_sum_int(bad);
  if (lane == 0) {
    s_d[wid][0] = wmin_w;
    s_d[wid][1] = wmax_w;
    s_d[wid][2] = q0;
    s_d[wid][3] = 0.0;
    s_i[wid][0] = npos;
    s_i[wid][1] = bad;
  }
  __syncthreads();
  if (tid == 0) {
    double wmin = s_d[0][0], wmax = s_d[0][1];
    for (int i = 1; i < kEsWaves; ++i) {
      wmin = fmin(wmin, s_d[i][0]);
      wmax = fmax(wmax, s_d[i][1]);
    }
    double a = 0.0;
    int n = 0, bd = 0;
    for (int i = 0; i < kEsWaves; ++i) {
      a += s_d[i][2];
      n += s_i[i][0];
      bd |= s_i[i][1];
    }
    EsTile o;
    o.wmin = wmin;
    o.wmax = wmax;
    o.q0 = a;
    o.pad0 = 0.0;
    o.npos = n;
    o.bad = bd != 0;
    o.kt = 0;
    o.nw = 0;
    o.wide = 1;
    o.small = 0;
    o.pad[0] = o.pad[1] = 0;
    if (n > 0) es_window(wmin, wmax, o.kt, o.nw);
    *rec = o;
    s_dec[0] = o.kt;
    s_dec[1] = o.nw;
    s_dec[2] = 0;  // no scaling in fp64
    s_dec[3] = (!o.bad && n > 0) ? 1 : 0;
  }
  __syncthreads();
  if (!s_dec[3]) return;
  const int kt = s_dec[0], nw = s_dec[1], tau = s_dec[2];
  const int npad = (nw + 15) / 16 * 16;
  for (int k = tid; k < npad; k += kEsThreads) s_rate[k] = (k < nw) ? es_rate<Real>(kt + 1 + k, tau) : (Real)1;
  // the expansion's variable u = a_kt w (scaled units) is at most 1/4 on this tile
  const Real a_kt = (Real)ldexp(exp((double)kt * kEsStep), -tau);
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
  const int M = (n + kEsThreads - 1) / kEsThreads;
  for (int j = n + tid; j < M * kEsThreads; j += kEsThreads) {  // padding entries contribute 0
    s_w[j] = (Real)0;
    s_q[j] = 0.0f;
  }
  __syncthreads();
  {
    // power sums T_j = sum q u^j of the tile (1/j! applied when they are used)
    Real T[kEsTaylor];
#pragma unroll
    for (int j = 0; j < kEsTaylor; ++j) T[j] = (Real)0;
    for (int m = 0; m < M; ++m) {
      const int j = tid + m * kEsThreads;
      const Real u = a_kt * s_w[j];
      Real pw = (Real)s_q[j];
#pragma unroll
      for (int i = 0; i < kEsTaylor; ++i) {
        T[i] += pw;
        pw *= u;
      }
    }
    const Real tot = wave_reduce_scatter<kEsTaylor, Real>(T, lane);
    if ((lane & (64 / kEsTaylor - 1)) == 0) s_tay[wid][lane / (64 / kEsTaylor)] = tot;
  }
  int nb = 0;
  for (; nb + 16 <= nw; nb += 16) es_moments_block<16, Real>(s_w, s_q, s_rate, M, nb, tid, lane, wid, s_red);
  if (nb + 8 <= nw) {
    es_moments_block<8, Real>(s_w, s_q, s_rate, M, nb, tid, lane, wid, s_red);
    nb += 8;
  }
  for (; nb < nw; nb += 4) es_moments_block<4, Real>(s_w, s_q, s_rate, M, nb, tid, lane, wid, s_red);
  __syncthreads();
  for (int k = tid; k < nw; k += kEsThreads) {
    Real s = s_red[0][k];
#pragma unroll
    for (int i = 1; i < kEsWaves; ++i) s += s_red[i][k];
    part[kEsTaylor + k] = (double)s;
  }
  if (tid < kEsTaylor) {
    Real s = s_tay[0][tid];
#pragma unroll
    for (int i = 1; i < kEsWaves; ++i) s += s_tay[i][tid];
    part[tid] = (double)s;
  }
}

// ------------------------------------------------------------------ moments (fp32)
// Persistent workgroups walk the (row, tile, law) records; while one tile is
// summed the next one's p and q are in flight.  Per tile: statistics and the
// record, a stable counting sort of the positive-weight tokens by binary
// exponent into LDS, then runs of 512 consecutive sorted tokens (two per wave):
// each run takes exponentials only on its own window [kt_r + 1, kt_r + nw_r]
// and power sums at its own expansion node kt_r; a run's power sums are turned
// into the tile's nodes kt + 1 .. kt_r and moved to the tile's expansion node
// kt (u = a_kt w <= a_kt_r w <= 1/4).  The tile record is the one the fp64 tile
// path writes: power sums at kt, moments of the nodes kt + 1 .. kt + nw.
constexpr int kEsRun = 512;             // sorted tokens per run
constexpr int kEsRunPer = kEsRun / 64;  // per lane
constexpr int kEsWin32 = 240;           // window bound of an fp32 tile: a span within 2^161 needs <= 233 nodes

// Node rates of fp32 tiles: log2(e) a_k = log2(e) e^(k/2) as an fp32 mantissa
// in [1, 2) and a binary exponent, for every node an fp32 tile can reach
// (ratios in the fp32 normal range: -181 <= kt, window top <= 180, plus the
// three filler nodes of a last block of four).  Built at compile time: e^(1/2)
// from its series, then successive products and quotients (relative error
// below 1e-13 over the range), rounded once to fp32.
constexpr int kEsNodeLo = -192, kEsNodeHi = 192;
struct EsRateTab {
  float mant[kEsNodeHi - kEsNodeLo];
  int expo[kEsNodeHi - kEsNodeLo];
};
constexpr EsRateTab es_make_rate_tab() {
  EsRateTab t{};
  double eh = 1.0, term = 1.0;
  for (int i = 1; i < 24; ++i) {
    term *= 0.5 / i;
    eh += term;
  }
  for (int dir = 0; dir < 2; ++dir) {
    double v = kEsLog2e;
    for (int k = 0; dir == 0 ? k < kEsNodeHi : k >= kEsNodeLo; k += dir == 0 ? 1 : -1) {
      double x = v;
      int n = 0;
      while (x >= 2.0) {
        x *= 0.5;
        ++n;
      }
      while (x < 1.0) {
        x *= 2.0;
        --n;
      }
      t.mant[k - kEsNodeLo] = (float)x;
      t.expo[k - kEsNodeLo] = n;
      v = dir == 0 ? v * eh : v / eh;
    }
  }
  return t;
}
__constant__ EsRateTab kEsRates = es_make_rate_tab();

// log2(e) a_k 2^-tau in fp32 for a uniform node k: scalar loads and an integer
// add to the exponent field (the scaled rates of a tile's nodes are normal:
// a_k w lies within [2^-160, 22] on the window and w 2^tau within 2^+-81).
__device__ __forceinline__ float es_rate_f32(int k, int tau) {
  const int i = min(max(k - kEsNodeLo, 0), kEsNodeHi - kEsNodeLo - 1);
  return __int_as_float(__float_as_int(kEsRates.mant[i]) + ((kEsRates.expo[i] - tau) << 23));
}

// A load through the scalar cache (constant address space) at a wave-uniform
// address: it waits on the scalar counter, so vector loads in flight (the next
// tile's p and q) are not waited for.  Only for data no kernel in flight writes.
template <typename T>
__device__ __forceinline__ T es_sload(const T* p) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);  // the address is the same in every lane: say so
  const uint64_t u = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                     (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
  return *(const __attribute__((address_space(4))) T*)(u);
}
// a whole record, dword by dword (merged into wide scalar loads; the scalar unit
// has no 12-byte load, so a partial read of a record would go to the vector unit)
template <typename T>
__device__ __forceinline__ T es_sload_rec(const T* p) {
  static_assert(sizeof(T) % 16 == 0, "whole 16-byte pieces");
  uint32_t raw[sizeof(T) / 4];
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) raw[i] = es_sload(reinterpret_cast<const uint32_t*>(p) + i);
  T out;
  __builtin_memcpy(&out, raw, sizeof(T));
  return out;
}


// Workgroup barrier that orders LDS only: global loads issued before it stay in flight.
__device__ __forceinline__ void es_lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Batcher's odd-even merge sort of N keys held by one lane (N a power of two):
// a fixed network of compare-exchanges on compile-time indices.
template <int N>
__device__ __forceinline__ void es_lane_sort(uint32_t (&k)[N]) {
#pragma unroll
  for (int p = 1; p < N; p <<= 1) {
#pragma unroll
    for (int d = p; d >= 1; d >>= 1) {
#pragma unroll
      for (int j = d % p; j + d < N; j += 2 * d) {
#pragma unroll
        for (int i = 0; i < d; ++i) {
          const int a = i + j, b = i + j + d;
          if (b < N && (a / (2 * p)) == (b / (2 * p))) {
            const uint32_t x = k[a], y = k[b];
            k[a] = min(x, y);
            k[b] = max(x, y);
          }
        }
      }
    }
  }
}

// NB window nodes of a run: sum over the run's tokens of q exp(-a_k w), added to
// the wave's moments (nodes at or above lim are not written).
template <int NB, int E>
__device__ __forceinline__ void es_run_block(const float (&w)[E], const float (&qq)[E], const float* __restrict__ rate,
                                             int lane, float* __restrict__ red, int lim) {
  float rt[NB], acc[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    rt[i] = rate[i];
    acc[i] = 0.0f;
  }
#pragma unroll
  for (int e = 0; e < E; ++e) {
#pragma unroll
    for (int i = 0; i < NB; ++i) acc[i] = fmaf(qq[e], es_decay(rt[i], w[e]), acc[i]);
  }
  const float tot = wave_reduce_scatter_f32<NB>(acc, lane);
  const int node = es_scatter_node<NB>(lane);
  if (es_scatter_writer<NB>(lane) && node < lim) red[node] += tot;
}

// One run (wave-level): LDS rows 2r and 2r + 1 of the tile (512 tokens; the
// entries of tokens left out are zero).  red / tay: the wave's moments of the
// tile window and power sums at the tile's expansion node.
__device__ void es_moments_run(const float* __restrict__ s_w, const float* __restrict__ s_q,
                               const float* __restrict__ s_rate, int r, int kt, int nw, int tau, bool whole,
                               int lane, float* __restrict__ red, float* __restrict__ tay) {
  constexpr float kInvFact[kEsTaylor] = {1.0f,        1.0f,         0.5f,          1.0f / 6.0f,
                                         1.0f / 24.0f, 1.0f / 120.0f, 1.0f / 720.0f, 1.0f / 5040.0f};
  float w[kEsRunPer], qq[kEsRunPer];
  // the run's weight range on the weights' bit patterns (every w here is +0 or a positive
  // normal, so unsigned order is float order)
  uint32_t lo_u = 0x7F800000u, hi_u = 0u;  // +inf, +0
#pragma unroll
  for (int e = 0; e < kEsRunPer; ++e) {
    const int j = r * kEsRun + e * 64 + lane;
    w[e] = s_w[j];
    qq[e] = s_q[j];
  }
  if (whole) {
    // every entry is a token and each column is sorted: entry e (row 2r) <= entry e + 4 (row 2r + 1)
#pragma unroll
    for (int e = 0; e < kEsRunPer / 2; ++e) {
      lo_u = min(lo_u, __float_as_uint(w[e]));
      hi_u = max(hi_u, __float_as_uint(w[e + kEsRunPer / 2]));
    }
  } else {
#pragma unroll
    for (int e = 0; e < kEsRunPer; ++e) {
      hi_u = max(hi_u, __float_as_uint(w[e]));  // entries left out hold w = q = 0
      lo_u = (qq[e] > 0.0f) ? min(lo_u, __float_as_uint(w[e])) : lo_u;
    }
  }
  const float lo = __uint_as_float(__builtin_amdgcn_readfirstlane(es_wave_ext_u<false>(lo_u)));
  const float hi = __uint_as_float(__builtin_amdgcn_readfirstlane(es_wave_ext_u<true>(hi_u)));
  if (!(hi > 0.0f)) return;  // uniform: an empty run
  int ktr, nwr;
  es_window_f32(ldexpf(lo, -tau), ldexpf(hi, -tau), ktr, nwr);
  ktr = __builtin_amdgcn_readfirstlane(ktr);
  nwr = __builtin_amdgcn_readfirstlane(nwr);
  const int o = min(max(ktr - kt, 0), nw);                 // the run expands at node kt + o
  const int cnt = max(0, min(ktr + nwr, kt + nw) - (kt + o));  // then exponentials on kt + o + 1 .. kt + o + cnt
  // power sums at u = a'_(kt+o) w
  const float akt = s_rate[o] * (float)(1.0 / kEsLog2e);
  float T[kEsTaylor];
#pragma unroll
  for (int j = 0; j < kEsTaylor; ++j) T[j] = 0.0f;
#pragma unroll
  for (int e = 0; e < kEsRunPer; ++e) {
    const float u = akt * w[e];
    float pw = qq[e];
#pragma unroll
    for (int j = 0; j < kEsTaylor; ++j) {
      T[j] += pw;
      pw *= u;
    }
  }
  const float tt = wave_reduce_scatter_f32<kEsTaylor>(T, lane);
  float Tj[kEsTaylor];  // uniform: read from the lane that holds each sum (node 4 b2 + 2 b3 + b4)
#pragma unroll
  for (int j = 0; j < kEsTaylor; ++j)
    Tj[j] = __int_as_float(
        __builtin_amdgcn_readlane(__float_as_int(tt), 4 * ((j >> 2) & 1) + 8 * ((j >> 1) & 1) + 16 * (j & 1)));
  // window nodes
  int nb = 0;
  const float* rate = s_rate + o + 1;
  for (; nb + 16 <= cnt; nb += 16) es_run_block<16>(w, qq, rate + nb, lane, red + o + nb, 16);
  if (nb + 8 <= cnt) {
    es_run_block<8>(w, qq, rate + nb, lane, red + o + nb, 8);
    nb += 8;
  }
  if (nb + 4 <= cnt) {
    es_run_block<4>(w, qq, rate + nb, lane, red + o + nb, 4);
    nb += 4;
  }
  if (nb + 2 <= cnt) {
    es_run_block<2>(w, qq, rate + nb, lane, red + o + nb, 2);
    nb += 2;
  }
  if (nb < cnt) es_run_block<1>(w, qq, rate + nb, lane, red + o + nb, 1);
  // tile nodes kt + 1 .. kt + o from the run's expansion: node kt + 1 + i has a_k / a_(kt+o) = e^(-(o - 1 - i) h)
  for (int i = lane; i < o; i += 64) {
    const float v = __builtin_amdgcn_exp2f(-(float)(o - 1 - i) * (float)(kEsStep * kEsLog2e));
    float s = Tj[kEsTaylor - 1] * kInvFact[kEsTaylor - 1];
#pragma unroll
    for (int j = kEsTaylor - 2; j >= 0; --j) s = fmaf(s, -v, Tj[j] * kInvFact[j]);
    red[i] += s;
  }
  // the run's power sums at the tile's expansion node: T_j (a_kt / a_(kt+o))^j
  if (es_scatter_writer<kEsTaylor>(lane)) {
    const int j = es_scatter_node<kEsTaylor>(lane);
    tay[j] += __builtin_amdgcn_exp2f(-(float)(o * j) * (float)(kEsStep * kEsLog2e)) * tt;
  }
}

__device__ __forceinline__ void es_load_tile(const float* __restrict__ p, const float* __restrict__ q1,
                                             const float* __restrict__ q2, int64_t V, int64_t b, int t, int l,
                                             int tid, float (&pv)[kEsMomPer], float (&qv)[kEsMomPer]) {
  const int64_t off = b * V + (int64_t)t * kEsMomTile + tid;
  const float* pb = p + off;
  const float* qb = (l == 0 ? q1 : q2) + off;
  if ((int64_t)t * kEsMomTile + kEsMomTile <= V) {  // uniform: a whole tile
#pragma unroll
    for (int i = 0; i < kEsMomPer; ++i) {
      pv[i] = pb[i * kEsThreads];
      qv[i] = qb[i * kEsThreads];
    }
  } else {
    const int64_t rest = V - (int64_t)t * kEsMomTile - tid;
#pragma unroll
    for (int i = 0; i < kEsMomPer; ++i) {
      const bool in = i * kEsThreads < rest;
      pv[i] = in ? pb[i * kEsThreads] : 0.0f;
      qv[i] = in ? qb[i * kEsThreads] : 0.0f;
    }
  }
}

// G = B * T1 * L records, record g = (b * T1 + t) * L + l; workgroup w takes the
// records [w per, (w + 1) per).  status_set (nullable): row b's status word is set
// to 0 with its first record (the kernels after this one OR the row's flags into it).
__global__ __launch_bounds__(kEsThreads, 4) void es_moments_kernel(const float* __restrict__ p,
                                                                 const float* __restrict__ q1,
                                                                 const float* __restrict__ q2, int64_t V, int L,
                                                                 int64_t G, int per, EsWork es,
                                                                 int32_t* __restrict__ status_set) {
  __shared__ float s_w[kEsMomTile];
  __shared__ float s_q[kEsMomTile];
  __shared__ float s_red[kEsWaves][kEsWin32];
  __shared__ float s_tay[kEsWaves][kEsTaylor];
  __shared__ float s_rate[kEsWin32 + 5];  // log2(e) a_k 2^-tau for the nodes kt .. kt + nw + 4
  __shared__ float s_f[2][kEsWaves][2];  // by tile parity: the tile may be skipped without another barrier
  __shared__ double s_q0[2][kEsWaves];
  __shared__ int s_i[2][kEsWaves][2];
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);

  float pv[kEsMomPer], qv[kEsMomPer];
  const int64_t g0 = (int64_t)blockIdx.x * per, g1 = min(g0 + per, G);
  if (g0 >= g1) return;
  int64_t b = g0 / (es.T1 * L);
  int t = (int)((g0 / L) % es.T1), l = (int)(g0 % L);
  es_load_tile(p, q1, q2, V, b, t, l, tid, pv, qv);
  for (int64_t g = g0, par = 0; g < g1; ++g, par ^= 1) {
    const bool more = g + 1 < g1;
    const bool whole = (int64_t)t * kEsMomTile + kEsMomTile <= V;
    if (status_set && t == 0 && l == 0 && tid == 0) status_set[b] = 0;
    if (++l == L) {  // (b, t, l) of the next record
      l = 0;
      if (++t == es.T1) {
        t = 0;
        ++b;
      }
    }
    // (1) ratios and statistics
    float wv[kEsMomPer];  // 0 for a token left out
    float wlo = INFINITY, whi = 0.0f;
    bool anyspec = false, anyzero = false;
    int npos = 0;
#pragma unroll
    for (int i = 0; i < kEsMomPer; ++i) {
      const float pp = pv[i], qq = qv[i];
      // NaN, -inf, negative normal or denormal, +inf (-0 is a zero probability); for q
      // also a positive denormal (its ratio is taken below)
      anyspec |= __builtin_amdgcn_classf(pp, 0x21F) | __builtin_amdgcn_classf(qq, 0x29F);
      const bool pos = pp > 0.0f && qq > 0.0f;
      anyzero |= qq > 0.0f && pp == 0.0f;
      const float w = pos ? es_ratio<float>(pp, qq) : 0.0f;
      wv[i] = w;
      wlo = fminf(wlo, pos ? w : INFINITY);
      whi = fmaxf(whi, w);  // w >= 0
      npos += pos;
    }
    bool anybad = false, anysmall = false;
    if (__builtin_amdgcn_ballot_w64(anyspec) != 0) {  // uniform and rare: a bad or a denormal probability
      __asm__ volatile("");  // keeps this path a branch (not computed for every token and selected)
      wlo = INFINITY;
      whi = 0.0f;
#pragma unroll
      for (int i = 0; i < kEsMomPer; ++i) {
        const float pp = pv[i], qq = qv[i];
        anybad |= __builtin_amdgcn_classf(pp, 0x21F) | __builtin_amdgcn_classf(qq, 0x21F);
        const bool small = es_denormal(qq) && pp > 0.0f;
        anysmall |= small;
        if (small) wv[i] = es_ratio_small_q(pp, qq);
        const bool pos = pp > 0.0f && qq > 0.0f;
        wlo = fminf(wlo, pos ? wv[i] : INFINITY);
        whi = fmaxf(whi, wv[i]);
      }
    }
    double q0w = 0.0;  // the draft mass on zero-weight tokens (p = 0 < q), in waves that hold one
    if (__builtin_amdgcn_ballot_w64(anyzero) != 0) {
      float q0f = 0.0f;
#pragma unroll
      for (int i = 0; i < kEsMomPer; ++i) q0f += (qv[i] > 0.0f && pv[i] == 0.0f) ? qv[i] : 0.0f;
      q0w = wave_sum((double)q0f);
    }
    wlo = es_wave_ext<false>(wlo);
    whi = es_wave_ext<true>(whi);
    npos = wave_sum_int(npos);
    const int bad = (__builtin_amdgcn_ballot_w64(anybad) != 0 ? 1 : 0) |
                    (__builtin_amdgcn_ballot_w64(anysmall) != 0 ? 2 : 0);  // bit 1: a denormal draft probability
    if (lane == 0) {
      s_f[par][wid][0] = wlo;
      s_f[par][wid][1] = whi;
      s_q0[par][wid] = q0w;
      s_i[par][wid][0] = npos;
      s_i[par][wid][1] = bad;
    }
    es_lds_barrier();
    // every thread combines the same values in the same order
    float wmin = s_f[par][0][0], wmax = s_f[par][0][1];
    double q0 = s_q0[par][0];
    int n = s_i[par][0][0], bd = s_i[par][0][1], smallq;
#pragma unroll
    for (int i = 1; i < kEsWaves; ++i) {
      wmin = fminf(wmin, s_f[par][i][0]);
      wmax = fmaxf(wmax, s_f[par][i][1]);
      q0 += s_q0[par][i];
      n += s_i[par][i][0];
      bd |= s_i[par][i][1];
    }
    smallq = (bd >> 1) & 1;
    bd &= 1;
    int kt = 0, nw = 0, tau = 0, wide = 0;
    if (n > 0) {
      if (!(wmin >= __FLT_MIN__) || !(wmax <= __FLT_MAX__)) {  // a weight that is not an fp32 normal
        wide = 1;
      } else {
        int range;
        es_scale_f32(wmin, wmax, tau, range);
        es_window_f32(wmin, wmax, kt, nw);
        wide = (range > kEsWideRange || nw > kEsWin32) ? 1 : 0;
      }
    }
    // the same in every lane: make it explicit (scalar registers, scalar table loads)
    kt = __builtin_amdgcn_readfirstlane(kt);
    nw = __builtin_amdgcn_readfirstlane(nw);
    tau = __builtin_amdgcn_readfirstlane(tau);
    n = __builtin_amdgcn_readfirstlane(n);
    if (tid == 0) {
      EsTile o;
      o.wmin = n > 0 ? (double)wmin : INFINITY;
      o.wmax = (double)wmax;
      o.pad0 = 0.0;
      o.q0 = q0;
      o.npos = n;
      o.bad = bd != 0;
      o.kt = wide ? 0 : kt;
      o.nw = wide ? 0 : nw;
      o.wide = wide;
      o.small = smallq;
      o.pad[0] = o.pad[1] = 0;
      es.tile[g] = o;
    }
    if (bd || n == 0 || wide) {  // uniform; an fp64 tile is taken by the coefficient kernel
      if (more) es_load_tile(p, q1, q2, V, b, t, l, tid, pv, qv);
      continue;
    }
    // (2) each thread sorts its tokens by weight (key: the weight's bits above the
    // last four, then the slot; tokens left out last) and the tile is laid out
    // rank by rank: LDS row i holds every thread's i-th smallest weight, so a run
    // (two rows) holds weights of nearby quantiles
    // here a token is in the sum exactly when its weight is positive (a weight that
    // is not an fp32 normal made the tile wide)
    uint32_t key[kEsMomPer];
#pragma unroll
    for (int i = 0; i < kEsMomPer; ++i) {
      const bool pos = wv[i] > 0.0f;
      key[i] = (pos ? (__float_as_uint(wv[i]) & ~15u) : ~15u) | (uint32_t)i;
      s_w[i * kEsThreads + tid] = ldexpf(wv[i], tau);  // this thread's column only
      s_q[i * kEsThreads + tid] = pos ? qv[i] : 0.0f;
    }
    es_lane_sort<kEsMomPer>(key);
    {
      float sw[kEsMomPer], sq[kEsMomPer];
#pragma unroll
      for (int i = 0; i < kEsMomPer; ++i) {
        const int from = (int)(key[i] & 15u) * kEsThreads + tid;
        sw[i] = s_w[from];
        sq[i] = s_q[from];
      }
#pragma unroll
      for (int i = 0; i < kEsMomPer; ++i) {
        s_w[i * kEsThreads + tid] = sw[i];
        s_q[i * kEsThreads + tid] = sq[i];
      }
    }
    for (int k = wid; k <= nw + 4; k += kEsWaves) {  // scalar table loads: the prefetch below is not waited for
      const float rt = es_rate_f32(kt + k, tau);
      if (lane == 0) s_rate[k] = rt;
    }
    for (int k = lane; k < nw; k += 64) s_red[wid][k] = 0.0f;
    if (lane < kEsTaylor) s_tay[wid][lane] = 0.0f;
    es_lds_barrier();
    if (more) es_load_tile(p, q1, q2, V, b, t, l, tid, pv, qv);  // in flight during the runs
    __asm__ volatile("" ::: "memory");  // keeps the loads here (not sunk past the runs)
    // (3) runs: rows 2r and 2r + 1
    const bool full = whole && n == kEsMomTile;  // every entry of the layout is a token
    for (int r = wid; r < kEsMomPer / 2; r += kEsWaves)
      es_moments_run(s_w, s_q, s_rate, r, kt, nw, tau, full, lane, s_red[wid], s_tay[wid]);
    es_lds_barrier();
    // (4) the tile's moments and power sums, waves in order
    double* part = es.part + g * kEsPart;
    for (int k = tid; k < nw; k += kEsThreads)
      part[kEsTaylor + k] = (double)(((s_red[0][k] + s_red[1][k]) + s_red[2][k]) + s_red[3][k]);
    if (tid < kEsTaylor) part[tid] = (double)(((s_tay[0][tid] + s_tay[1][tid]) + s_tay[2][tid]) + s_tay[3][tid]);
  }
}

// ------------------------------------------------------------------ evaluation (fp64)
// The fp64 path: one evaluation tile (2048 tokens) of a row with an fp64 tile,
// run by the coefficient kernel: r(y) = p(y) [P + sum over the tile's window of
// c_k exp(-a_k w(y))] + the zero-weight closed forms, P the expansion of the
// grid nodes below the window.
template <typename Real, int L>
__device__ bool es_eval_tile(const float* __restrict__ pb, const float* __restrict__ q1b,
                             const float* __restrict__ q2b, int64_t V, int K, int64_t t, float* __restrict__ rb,
                             const EsPlan& pl, const double* __restrict__ ctab) {
  static_assert(sizeof(Real) == 8, "the fp64 path");
  __shared__ Real s_w[kEsEvalTile];
  __shared__ uint16_t s_pos[kEsEvalTile];
  __shared__ Real s_acc[kEsEvalTile];
  // one LDS area: first the row's fp64 coefficients up to kt (for the expansion),
  // then the window's node rates and coefficients in the tile's precision
  __shared__ Real s_tab[2 * kEsMaxWin];
  static_assert(sizeof(Real) * 2 * kEsMaxWin >= sizeof(double) * kEsMaxNodes, "staging area");
  Real* const s_rate = s_tab;
  Real* const s_coef = s_tab + kEsMaxWin;
  double* const s_cf = reinterpret_cast<double*>(s_tab);
  __shared__ int s_wave[kEsWaves];
  __shared__ double s_d[kEsWaves][2][2];
  __shared__ int s_dec[2][3];  // per law: first row node of the window, window length, last expansion node
  __shared__ Real s_poly[kEsTaylor];
  __shared__ Real s_akt;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t base = t * kEsEvalTile;

  float pv[kEsEvalPer], qv[L][kEsEvalPer];
  Real wv[L][kEsEvalPer];
  bool pos[L][kEsEvalPer];
#pragma unroll
  for (int i = 0; i < kEsEvalPer; ++i) {
    const int64_t x = base + i * kEsThreads + tid;
    pv[i] = (x < V) ? pb[x] : 0.0f;
    qv[0][i] = (x < V) ? q1b[x] : 0.0f;
    if (L == 2) qv[L - 1][i] = (x < V) ? q2b[x] : 0.0f;
  }
  if (pl.nk > 0) {
    double wmin[2] = {INFINITY, INFINITY}, wmax[2] = {0.0, 0.0};
#pragma unroll
    for (int l = 0; l < L; ++l) {
      Real lo = (Real)INFINITY, hi = (Real)0;
#pragma unroll
      for (int i = 0; i < kEsEvalPer; ++i) {
        pos[l][i] = pv[i] > 0.0f && qv[l][i] > 0.0f;
        const Real w = pos[l][i] ? es_ratio<Real>(pv[i], qv[l][i]) : (Real)0;
        wv[l][i] = w;
        lo = pos[l][i] ? fmin(lo, w) : lo;
        hi = pos[l][i] ? fmax(hi, w) : hi;
      }
      wmin[l] = (double)es_wave_min(lo);
      wmax[l] = (double)es_wave_max(hi);
    }
    if (lane == 0) {
      for (int l = 0; l < L; ++l) {
        s_d[wid][l][0] = wmin[l];
        s_d[wid][l][1] = wmax[l];
      }
    }
    __syncthreads();
    if (tid == 0) {
      for (int l = 0; l < L; ++l) {
        for (int i = 0; i < kEsWaves; ++i) {
          wmin[l] = fmin(wmin[l], s_d[i][l][0]);
          wmax[l] = fmax(wmax[l], s_d[i][l][1]);
        }
      }
      for (int l = 0; l < L; ++l) {
        int i0 = pl.nk, cnt = 0, kt = pl.k_lo + pl.nk;
        if (wmax[l] > 0.0) {
          int nw;
          es_window(wmin[l], wmax[l], kt, nw);
          i0 = std::min(std::max(kt + 1 - pl.k_lo, 0), pl.nk);
          const int i1 = std::min(kt + nw - pl.k_lo, pl.nk - 1);
          cnt = std::max(0, i1 - i0 + 1);
        }
        s_dec[l][0] = i0;
        s_dec[l][1] = cnt;
        s_dec[l][2] = kt;
      }
    }
    __syncthreads();
  }
  constexpr int tau = 0;  // no scaling in fp64
#pragma unroll
  for (int i = 0; i < kEsEvalPer; ++i) s_acc[i * kEsThreads + tid] = (Real)0;
  if (pl.nk > 0) {
#pragma unroll
    for (int l = 0; l < L; ++l) {
      const int i0 = s_dec[l][0], cnt = s_dec[l][1], kt = s_dec[l][2];
      const double* c = ctab + l * kEsMaxWin;
      // expansion of the nodes up to kt: B_j = sum_(k <= kt) c_k (a_k / a_kt)^j, one thread per j,
      // nodes in ascending order from LDS; stored as B_j / j! in the tile's scale
      const int top = std::min(kt, pl.k_lo + pl.nk - 1);
      for (int k = pl.k_lo + tid; k <= top; k += kEsThreads) s_cf[k - pl.k_lo] = c[k - pl.k_lo];
      __syncthreads();
      if (tid < kEsTaylor) {
        const int j = tid;
        const double dj = exp(-(double)j * kEsStep);  // (a_(k-1) / a_k)^j
        double acc = 0.0;
        for (int k = pl.k_lo; k <= top; ++k) acc = acc * dj + s_cf[k - pl.k_lo];
        if (top >= pl.k_lo && kt > top) acc *= exp(-(double)j * (double)(kt - top) * kEsStep);
        s_poly[j] = (Real)ldexp(acc * es_inv_fact(j), -tau);
      }
      if (tid == 0) s_akt = (Real)ldexp(exp((double)kt * kEsStep), -tau);
      __syncthreads();  // the staging area becomes the window's tables
      for (int k = tid; k < cnt; k += kEsThreads) {
        s_rate[k] = es_rate<Real>(pl.k_lo + i0 + k, tau);
        s_coef[k] = (Real)ldexp(c[i0 + k], -tau);
      }
      int n = 0;
      int off = block_compact_offset<kEsEvalPer>(pos[l], s_wave, n);
#pragma unroll
      for (int i = 0; i < kEsEvalPer; ++i) {
        if (pos[l][i]) {
          s_w[off] = wv[l][i];
          s_pos[off] = (uint16_t)(i * kEsThreads + tid);
          ++off;
        }
      }
      __syncthreads();
      Real poly[kEsTaylor];
#pragma unroll
      for (int j = 0; j < kEsTaylor; ++j) poly[j] = s_poly[j];
      const Real akt = s_akt;
      for (int j0 = 0; j0 < n; j0 += 4 * kEsThreads) {
        Real w[4], acc[4];
        int ps[4];
        bool ok[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = j0 + e * kEsThreads + tid;
          ok[e] = j < n;
          w[e] = ok[e] ? s_w[j] : (Real)0;
          ps[e] = ok[e] ? (int)s_pos[j] : 0;
          acc[e] = (Real)0;
        }
        int k = 0;
        for (; k + 16 <= cnt; k += 16) {
          Real blk[4] = {(Real)0, (Real)0, (Real)0, (Real)0};
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const Real rt = s_rate[k + i], cf = s_coef[k + i];
#pragma unroll
            for (int e = 0; e < 4; ++e) blk[e] = es_fma(cf, es_decay(rt, w[e]), blk[e]);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += blk[e];
        }
        {
          Real blk[4] = {(Real)0, (Real)0, (Real)0, (Real)0};
          for (; k < cnt; ++k) {
            const Real rt = s_rate[k], cf = s_coef[k];
#pragma unroll
            for (int e = 0; e < 4; ++e) blk[e] = es_fma(cf, es_decay(rt, w[e]), blk[e]);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            // far nodes: sum_j (-u)^j B_j / j!, u = a_kt w <= 1/4 (Horner)
            const Real nu = -akt * w[e];
            Real pe = poly[kEsTaylor - 1];
#pragma unroll
            for (int j = kEsTaylor - 2; j >= 0; --j) pe = es_fma(pe, nu, poly[j]);
            acc[e] += blk[e] + pe;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (ok[e]) s_acc[ps[e]] += acc[e];  // one entry per token and law: no two threads share a slot
      }
      __syncthreads();  // tables and the compacted list are rebuilt for the next law; s_acc is read below
    }
  }
  const double q0a = pl.q0[0], q0b = (L == 2) ? pl.q0[1] : 0.0;
  double zw = q0a;  // K i.i.d. drafts: Q0^(K-1)
  for (int j = 2; j < K; ++j) zw *= q0a;
#pragma unroll
  for (int i = 0; i < kEsEvalPer; ++i) {
    const int64_t x = base + i * kEsThreads + tid;
    if (x >= V) break;
    const float pp = pv[i];
    const Real acc = s_acc[i * kEsThreads + tid];
    const float quad = (float)((double)pp * (double)acc);
    float v = 0.0f;
    if (L == 1) {
      const float qq = qv[0][i];
      if (qq > 0.0f) v = (pp > 0.0f) ? ((K == 2) ? fmaf(2.0f * qq, (float)q0a, quad) : quad) : (float)((double)qq * zw);
    } else {
      // two laws: a zero-weight pole of the other draft adds q_i(y) Qj_0; a zero target splits it in half
      const float a = qv[0][i], c = qv[L - 1][i];
      const float za = (a > 0.0f) ? a * (float)q0b : 0.0f, zc = (c > 0.0f) ? c * (float)q0a : 0.0f;
      v = (pp > 0.0f) ? quad + za + zc : 0.5f * (za + zc);
    }
    rb[x] = v;
  }
  return true;
}

// ------------------------------------------------------------------ evaluation (fp32)
// Persistent workgroups over the (row, tile) pairs of 1024 tokens, the next
// tile's p and q in flight meanwhile.  Every query token takes its own nodes:
// with k0 its first node where a_k w > 1/4, the nine nodes k0 .. k0 + 8 have
// a_k w in (1/4, 22.5], the grid nodes below k0 enter through the expansion
// sum_j B_j(k0 - 1) (-a_(k0-1) w)^j / j!, B_j(k) = sum over grid nodes k' <= k
// of c_k' (a_k' / a_k)^j, and the nodes above k0 + 8 (a_k w > 22) are dropped.
// Since x = a_k0 w lies in (1/4, e^(1/2)/4], the nine node terms and the
// expansion together are one function of x per node row, kept as a polynomial
// of degree 10 in t = (x - x_mid) / delta (coefficients from the coefficient
// kernel; the node terms by Chebyshev interpolation, the expansion exactly).
// Per tile and law two LDS tables, in the tile's scale, are indexed by
// d = k0 - 1 - kt (kt: the tile's first expansion node): the polynomial rows
// and the node rates; each token reads them at its own offset.
constexpr int kEsTokNodes = kEsTokNodesC;       // node terms per query token
constexpr int kEsTokPer = 4;                    // tokens per thread
constexpr int kEsTokTile = kEsThreads * kEsTokPer;  // 1024 tokens per tile
constexpr int kEsTabRows = kEsWin32 + 1;        // d = 0 .. 240
constexpr int kEsPolyStride = 12;               // a polynomial row padded to three 16-byte LDS reads
static_assert(kEsPolyLen <= kEsPolyStride && kEsPolyStride % 4 == 0, "polynomial row layout");

template <int L>
__device__ __forceinline__ void es_load_eval(const float* __restrict__ p, const float* __restrict__ q1,
                                             const float* __restrict__ q2, int64_t V, int64_t b, int t, int tid,
                                             float (&pv)[kEsTokPer], float (&qv)[L][kEsTokPer]) {
  const int64_t off = b * V + (int64_t)t * kEsTokTile + tid;
  const float* pb = p + off;
  const float* qa = q1 + off;
  const float* qc = ((L == 2) ? q2 : q1) + off;
  if ((int64_t)t * kEsTokTile + kEsTokTile <= V) {  // uniform: a whole tile
#pragma unroll
    for (int i = 0; i < kEsTokPer; ++i) {
      pv[i] = pb[i * kEsThreads];
      qv[0][i] = qa[i * kEsThreads];
      if (L == 2) qv[L - 1][i] = qc[i * kEsThreads];
    }
  } else {
    const int64_t rest = V - (int64_t)t * kEsTokTile - tid;
#pragma unroll
    for (int i = 0; i < kEsTokPer; ++i) {
      const bool in = i * kEsThreads < rest;
      pv[i] = in ? pb[i * kEsThreads] : 0.0f;
      qv[0][i] = in ? qa[i * kEsThreads] : 0.0f;
      if (L == 2) qv[L - 1][i] = in ? qc[i * kEsThreads] : 0.0f;
    }
  }
}

// Residual sums of Algorithm 1 (kRes): per 1024-token tile, each wave's fp64 sum of
// max(0, p - r) over its 256 tokens (r as stored), at rsum[(b nsub + tile) 4 + wave]
// (NaN where a p or r is not a probability).
__device__ __forceinline__ void es_residual_sums(const float (&pc)[kEsTokPer], const float (&rc)[kEsTokPer],
                                                 double* __restrict__ rsum, int64_t b, int64_t tile, int64_t nsub,
                                                 int lane, int wid) {
  double local = 0.0;
  bool bad = false;
#pragma unroll
  for (int i = 0; i < kEsTokPer; ++i) {
    bad |= bad_prob(pc[i]) || bad_prob(rc[i]);
    local += residual_of(pc[i], rc[i]);
  }
  const double tot = wave_sum_dpp(local);
  const bool any_bad = __builtin_amdgcn_ballot_w64(bad) != 0;
  if (lane == 0) rsum[(b * nsub + tile) * kEsWaves + wid] = any_bad ? (double)NAN : tot;
}

// Workgroup w takes the tiles [w per, (w + 1) per) of the B * T2 (row, tile)
// pairs, row-major.  A tile's weight range comes from the moments record of
// the 4096-token tile that holds it, so evaluation needs no statistics pass.
// kRes: the residual sums of Algorithm 1 are written too (rsum).
template <int L, bool kRes>
__global__ __launch_bounds__(kEsThreads) void es_eval_kernel(const float* __restrict__ p,
                                                              const float* __restrict__ q1,
                                                              const float* __restrict__ q2, int64_t V, int K,
                                                              float* __restrict__ r, int64_t G, int per, EsWork es,
                                                              double* __restrict__ rsum, int64_t nsub) {
  static_assert(kEsMomTile % kEsTokTile == 0, "an evaluation tile lies in one moments tile");
  __shared__ __align__(16) float s_a[L][kEsTabRows * kEsPolyStride];  // A_n(k0 = kt + 1 + d) 2^-tau
  __shared__ float s_r[L][kEsTabRows];                                // log2(e) a_(kt+1+d) 2^-tau
  const int tid = threadIdx.x;
  // t = (a_k0 w - x_mid) / delta from x = log2(e) a_k0 w
  constexpr float kTs = (float)(1.0 / (kEsPolyDelta * kEsLog2e)), kTo = (float)(-kEsPolyXm / kEsPolyDelta);

  const int64_t g0 = (int64_t)blockIdx.x * per, g1 = min(g0 + per, G);
  if (g0 >= g1) return;
  int64_t b = __builtin_amdgcn_readfirstlane((int)(g0 / es.T3));  // rows < 2^31
  int t = __builtin_amdgcn_readfirstlane((int)(g0 - b * es.T3));
  int64_t built = -1;  // moments record whose tables are in LDS (both halves of it share them)
  int tau = 0, kt[2] = {0, 0}, D[2] = {-1, -1}, smallq[2] = {0, 0};
  float pv[kEsTokPer], qv[L][kEsTokPer];
  es_load_eval<L>(p, q1, q2, V, b, t, tid, pv, qv);
  for (int64_t g = g0; g < g1; ++g) {
    const int64_t base = (int64_t)t * kEsTokTile;
    const bool whole = base + kEsTokTile <= V;
    float* rb = r + b * V + base + tid;  // (b, t) is this tile until advanced below
    float pc[kEsTokPer], qc[L][kEsTokPer];
#pragma unroll
    for (int i = 0; i < kEsTokPer; ++i) {
      pc[i] = pv[i];
#pragma unroll
      for (int l = 0; l < L; ++l) qc[l][i] = qv[l][i];
    }
    const int64_t bb = __builtin_amdgcn_readfirstlane((int)b);  // uniform: scalar loads below
    const int tt = __builtin_amdgcn_readfirstlane(t);
    if (++t == es.T3) {
      t = 0;
      ++b;
    }
    const EsPlan pl = es_sload_rec(es.plan + bb);
    const int flags = pl.flags, fp64 = pl.fp64, k_lo = pl.k_lo, nk = pl.nk;
    if (flags || fp64) {  // uniform; a row in fp64 is evaluated by the coefficient kernel
      if (g + 1 < g1) es_load_eval<L>(p, q1, q2, V, b, t, tid, pv, qv);
      if (flags) {
#pragma unroll
        for (int i = 0; i < kEsTokPer; ++i)
          if (whole || base + i * kEsThreads + tid < V) rb[i * kEsThreads] = NAN;
      }
      if (kRes) {  // the residual sums from the r written (a flagged row: NaN)
        float rc[kEsTokPer];
#pragma unroll
        for (int i = 0; i < kEsTokPer; ++i)
          rc[i] = flags ? NAN : ((whole || base + i * kEsThreads + tid < V) ? rb[i * kEsThreads] : 0.0f);
        es_residual_sums(pc, rc, rsum, bb, tt, nsub, tid & 63, tid >> 6);
      }
      continue;
    }
    float acc[kEsTokPer];
#pragma unroll
    for (int i = 0; i < kEsTokPer; ++i) acc[i] = 0.0f;
    if (nk <= 0) tau = 0;
    const int64_t recno = bb * es.T1 + tt / (kEsMomTile / kEsTokTile);
    if (nk > 0 && recno != built) {  // uniform
      // (1) the tile's scale and tables from the moments records (every record of a
      // row without an fp64 tile has its ratios in the fp32 normal range)
      if (built >= 0) es_lds_barrier();  // every wave is done with the previous tables
      built = recno;
      float wmin[2], wmax[2];
#pragma unroll
      for (int l = 0; l < L; ++l) {
        const EsTile rec = es_sload_rec(es.tile + recno * L + l);
        wmin[l] = (float)rec.wmin;  // +inf / 0 when the law has no positive weight here
        wmax[l] = (float)rec.wmax;
        smallq[l] = rec.small;
      }
      const float lo = fminf(wmin[0], wmin[L - 1]), hi = fmaxf(wmax[0], wmax[L - 1]);
      int range = 0;
      tau = 0;
      if (hi > 0.0f) es_scale_f32(lo, hi, tau, range);
#pragma unroll
      for (int l = 0; l < L; ++l) {
        kt[l] = 0;
        D[l] = -1;
        if (!(wmax[l] > 0.0f)) continue;  // uniform
        int nw, ktlo;
        es_window_f32(wmin[l], wmax[l], kt[l], nw);
        es_window_f32(wmin[l], wmin[l], ktlo, nw);  // the last expansion node of the smallest weight
        D[l] = min(max(ktlo - kt[l], 0), kEsTabRows - 1);
        // tables: every thread loads its entries (vector loads, all in flight at once); the
        // coefficient kernel wrote the rows [0, nrow) that the row's tokens of either law can
        // reach (a row before the grid, i < 0, would be a node range no token takes)
        const double* at = es.atab + (bb * L + l) * (int64_t)kEsAtabRows * kEsPolyLen;
        const int nrow = pl.nrow;
        for (int e = tid; e < (D[l] + 1) * kEsPolyStride; e += kEsThreads) {
          const int d = e / kEsPolyStride, n = e % kEsPolyStride, i = kt[l] + 1 + d - k_lo;
          const double v = (n < kEsPolyLen && i >= 0 && i < nrow) ? at[i * kEsPolyLen + n] : 0.0;
          s_a[l][e] = (float)ldexp(v, -tau);
        }
        for (int d = tid; d <= D[l]; d += kEsThreads) s_r[l][d] = es_rate_f32(kt[l] + 1 + d, tau);
      }
      es_lds_barrier();
    }
    // the next tile's p and q: issued after the table loads, so that waiting for those
    // never waits for these; in flight through this tile's arithmetic
    if (g + 1 < g1) es_load_eval<L>(p, q1, q2, V, b, t, tid, pv, qv);
    __asm__ volatile("" ::: "memory");
    if (nk > 0) {
      // (2) per token: the polynomial of its node row
#pragma unroll
      for (int l = 0; l < L; ++l) {
        if (D[l] < 0) continue;  // uniform
        const float* sa = s_a[l];
        const float* sr = s_r[l];
        // branch-free over the thread's tokens, so that their dependency chains interleave;
        // a token without a positive weight is evaluated at w = 1 and its result dropped
        bool ok[kEsTokPer];
        int d[kEsTokPer];
        float x[kEsTokPer];
        float ratio[kEsTokPer];
#pragma unroll
        for (int i = 0; i < kEsTokPer; ++i) {
          // no short-circuit and the ratio for every token (its inf or NaN for q = 0 is
          // selected away): straight-line code, no branches per token
          ok[i] = (pc[i] > 0.0f) & (qc[l][i] > 0.0f);
          ratio[i] = es_ratio<float>(pc[i], qc[l][i]);
        }
        if (smallq[l]) {  // uniform and rare: the moments record saw a denormal draft probability
          __asm__ volatile("");  // keeps this path a branch
#pragma unroll
          for (int i = 0; i < kEsTokPer; ++i)
            if (es_denormal(qc[l][i])) ratio[i] = es_ratio_small_q(pc[i], qc[l][i]);
        }
#pragma unroll
        for (int i = 0; i < kEsTokPer; ++i) {
          const float w = ok[i] ? ratio[i] : 1.0f;
          // d = kt(w) - kt, kt(w) = floor((ln 1/4 - ln w) / h)
          const float ktw =
              floorf(((float)kEsLnFar - __builtin_amdgcn_logf(w) * 0.69314718f) * (float)(1.0 / kEsStep));
          d[i] = min(max((int)ktw - kt[l], 0), D[l]);
          x[i] = sr[d[i]] * ldexpf(w, tau);  // log2(e) a_k0 w
        }
#pragma unroll
        for (int i = 0; i < kEsTokPer; ++i) {
          // Horner in t; the tokens of a thread interleave their chains
          const float tt = fmaf(x[i], kTs, kTo);
          const float4* pa = reinterpret_cast<const float4*>(sa + __umul24((unsigned)d[i], kEsPolyStride));
          const float4 a0 = pa[0], a1 = pa[1], a2 = pa[2];  // A_0 .. A_10 (a2.w: padding)
          float f = a2.z;
          f = fmaf(f, tt, a2.y);
          f = fmaf(f, tt, a2.x);
          f = fmaf(f, tt, a1.w);
          f = fmaf(f, tt, a1.z);
          f = fmaf(f, tt, a1.y);
          f = fmaf(f, tt, a1.x);
          f = fmaf(f, tt, a0.w);
          f = fmaf(f, tt, a0.z);
          f = fmaf(f, tt, a0.y);
          f = fmaf(f, tt, a0.x);
          acc[i] = (l == 0 ? 0.0f : acc[i]) + (ok[i] ? f : 0.0f);
        }
      }
    }
    // (3) epilogue: r(y) = p(y) 2^tau sum + the zero-weight closed forms; every form is
    // computed and then selected (kept in registers, so that the compiler does not turn
    // the selections into branches per token), and a whole tile stores without bounds tests
    const float q0a = (float)pl.q0[0], q0b = (L == 2) ? (float)pl.q0[1] : 0.0f;
    double zw = pl.q0[0];  // K i.i.d. drafts: Q0^(K-1)
    for (int j = 2; j < K; ++j) zw *= pl.q0[0];
    const float zwf = (float)zw;
    float out[kEsTokPer];
#pragma unroll
    for (int i = 0; i < kEsTokPer; ++i) {
      const float pp = pc[i];
      const float quad = ldexpf(pp * acc[i], tau);
      float v;
      if (L == 1) {
        const float qq = qc[0][i];
        float pos = (K == 2) ? fmaf(2.0f * qq, q0a, quad) : quad;
        float zero = qq * zwf;
        __asm__ volatile("" : "+v"(pos), "+v"(zero));
        v = (pp > 0.0f) ? pos : zero;
        v = (qq > 0.0f) ? v : 0.0f;
      } else {
        // two laws: a zero-weight pole of the other draft adds q_i(y) Qj_0; a zero target splits it in half
        const float a = qc[0][i], c = qc[L - 1][i];
        float za = (a > 0.0f) ? a * q0b : 0.0f, zc = (c > 0.0f) ? c * q0a : 0.0f;
        float pos = quad + za + zc, zero = 0.5f * (za + zc);
        __asm__ volatile("" : "+v"(pos), "+v"(zero));
        v = (pp > 0.0f) ? pos : zero;
      }
      out[i] = v;
    }
    if (whole) {
#pragma unroll
      for (int i = 0; i < kEsTokPer; ++i) rb[i * kEsThreads] = out[i];
    } else {
#pragma unroll
      for (int i = 0; i < kEsTokPer; ++i)
        if (base + i * kEsThreads + tid < V) rb[i * kEsThreads] = out[i];
    }
    if (kRes) es_residual_sums(pc, out, rsum, bb, tt, nsub, tid & 63, tid >> 6);  // tokens past V: p = r = 0
  }
}

// ------------------------------------------------------------------ coefficients
// Statistics of a row's tile records, merged in tile order.
struct EsMerge {
  double wmin[2], wmax[2], q0[2];  // per law
  int npos[2], bad, wide;          // wide: a tile to be taken in fp64
};

// Every wave reads the row's records itself (the same values in every lane), so
// that the merge and the plan need no reduction across lanes and no barrier.
template <int L>
__device__ EsMerge es_merge(const EsTile* __restrict__ rec, int64_t T1) {
  EsMerge m;
  m.wmin[0] = m.wmin[1] = INFINITY;
  m.wmax[0] = m.wmax[1] = 0.0;
  m.q0[0] = m.q0[1] = 0.0;
  m.npos[0] = m.npos[1] = 0;
  m.bad = m.wide = 0;
  constexpr int kB = 8;  // records whose loads are issued together
  for (int64_t t0 = 0; t0 < T1; t0 += kB) {
    double lo[kB][L], hi[kB][L], z[kB][L];
    int np[kB][L], bd[kB][L], wd[kB][L];
#pragma unroll
    for (int i = 0; i < kB; ++i)
#pragma unroll
      for (int l = 0; l < L; ++l) {
        const bool in = t0 + i < T1;
        const EsTile& e = rec[(in ? t0 + i : 0) * L + l];
        lo[i][l] = e.wmin;
        hi[i][l] = e.wmax;
        z[i][l] = e.q0;
        np[i][l] = in ? e.npos : 0;
        bd[i][l] = e.bad;
        wd[i][l] = e.wide;
        if (!in) {
          lo[i][l] = INFINITY;
          hi[i][l] = 0.0;
          z[i][l] = 0.0;
          bd[i][l] = wd[i][l] = 0;
        }
      }
#pragma unroll
    for (int i = 0; i < kB; ++i)
#pragma unroll
      for (int l = 0; l < L; ++l) {
        m.wmin[l] = fmin(m.wmin[l], lo[i][l]);
        m.wmax[l] = fmax(m.wmax[l], hi[i][l]);
        m.q0[l] += z[i][l];
        m.npos[l] += np[i][l];
        m.bad |= bd[i][l];
        m.wide |= wd[i][l] && !bd[i][l];
      }
  }
  return m;
}

// The row's plan from its merged records: flags, the grid's node range (the
// left-tail and right-tail cuts of the quadrature), fp64 evaluation.
template <int L>
__device__ EsPlan es_make_plan(const EsMerge& m, int K) {
  EsPlan pl;
  pl.flags = m.bad ? kRowBadProb : 0;
  pl.k_lo = 0;
  pl.nk = 0;
  pl.fp64 = m.wide ? 1 : 0;
  pl.q0[0] = m.q0[0];
  pl.q0[1] = m.q0[1];
  pl.nrow = 0;
  pl.pad_i = 0;
  for (int i = 0; i < 4; ++i) pl.pad[i] = 0.0;
  const bool any = (L == 1) ? m.npos[0] > 0 : (m.npos[0] > 0 && m.npos[1] > 0);
  if (!pl.flags && any) {
    double dmin, dmax;
    if (L == 1) {
      // K = 2 takes the zero-weight tokens in closed form; K >= 3 keeps them in S (denominator w(y) alone)
      dmin = (K == 2 || m.q0[0] == 0.0) ? K * m.wmin[0] : m.wmin[0];
      dmax = K * m.wmax[0];
    } else {
      dmin = m.wmin[0] + m.wmin[1];
      dmax = m.wmax[0] + m.wmax[1];
      int tau, range;
      es_scale(fmin(m.wmin[0], m.wmin[1]), fmax(m.wmax[0], m.wmax[1]), tau, range);
      if (range > kEsWideRange) pl.fp64 = 1;  // an evaluation tile mixes both laws' weights
    }
    const int k_lo = (int)floor((kEsLnEps - log(dmax)) / kEsStep);
    const int k_hi = (int)ceil((kEsLnLnInvEps - log(dmin)) / kEsStep);
    pl.k_lo = k_lo;
    pl.nk = k_hi - k_lo + 1;
    if (pl.nk > kEsMaxNodes) {  // only rows with probabilities far above 1 get here
      pl.flags = kRowRange;
      pl.nk = 0;
    } else {
      // polynomial rows of the evaluation: a query token with first window node k0 reads
      // row k0 - k_lo.  One law alone: k0 of the smallest weight lies before the grid's
      // end.  Two laws: a token of one law whose weight is far below the smallest
      // denominator w1 + w2 has k0 past the grid (every grid node enters through its
      // decayed expansion), so the rows run to the k0 of either law's smallest weight,
      // two rows to spare for the evaluation's fp32 logarithm.  Rows needing more than
      // the table holds (weights spanning far beyond the fp32 tiles' 2^160) go to fp64.
      int nrow = pl.nk + 16;
      for (int l = 0; l < L; ++l) nrow = max(nrow, (int)floor((kEsLnFar - log(m.wmin[l])) / kEsStep) + 3 - k_lo);
      if (nrow > kEsAtabRows) pl.fp64 = 1;
      pl.nrow = min(nrow, kEsAtabRows);
    }
  }
  if (pl.flags) pl.fp64 = 0;
  return pl;
}

// One workgroup per row, after the moments.  (1) Tiles the fp32 pass left
// aside are taken in fp64, in tile order.  (2) The tile records are merged in
// tile order (fp64): flags, zero-weight masses, the row's grid range.  (3) S_k
// from the tile windows, c_k and their prefix sums.  K i.i.d. drafts:
// c_k = K h a_k S_k^(K-1) (K >= 3 keeps the zero-weight mass Q0 in S); two
// laws: the queries of law 1 take h a_k S_k of law 2 and those of law 2 take
// h a_k S_k of law 1.  (4) A row with an fp64 tile (or, for two laws, weights
// spanning more than 2^160) is evaluated here in fp64.
template <int L>
__global__ __launch_bounds__(kEsThreads) void es_coef_kernel(const float* __restrict__ p,
                                                              const float* __restrict__ q1,
                                                              const float* __restrict__ q2, int64_t V, int K,
                                                              float* __restrict__ r, EsWork es,
                                                              int32_t* __restrict__ row_status) {
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t nrec = es.T1 * L;
  EsTile* rec = es.tile + b * nrec;
  double* part = es.part + b * nrec * kEsPart;
  const float* pb = p + b * V;
  __shared__ double s_c[L][kEsMaxWin];
  __shared__ double s_rho[kEsMaxWin];  // e^(-m h): (a_k / a_kt) for k = kt - m
  constexpr int kCh = 64;              // tile records staged per pass of (3)
  __shared__ __align__(16) int s_rkt[kCh];
  __shared__ __align__(16) int s_rnw[kCh];
  __shared__ double s_pow[kCh][kEsTaylor];
  // a chunk of records: window starts and lengths, power sums / j!; read after a barrier
  auto stage = [&](int64_t c0) {
    const int nc = (int)min((int64_t)kCh, nrec - c0);
    if (tid < nc) {
      const EsTile& e = rec[c0 + tid];
      s_rkt[tid] = e.kt;
      s_rnw[tid] = (e.npos > 0 && !e.bad) ? e.nw : -1;  // -1: the record adds nothing
    }
    for (int x = tid; x < nc * kEsTaylor; x += kEsThreads) {
      const int i = x / kEsTaylor, j = x % kEsTaylor;
      s_pow[i][j] = part[(c0 + i) * kEsPart + j] * es_inv_fact(j);
    }
  };

  // (1) the first chunk's loads go out first; the node ratios are computed meanwhile.
  // Every wave merges the records (tile order) and takes the plan from them; fp64
  // tiles (rare) are computed here, and the records are then read again.
  stage(0);
  for (int m = tid; m < kEsMaxWin; m += kEsThreads) s_rho[m] = exp(-(double)m * kEsStep);
  EsMerge mg = es_merge<L>(rec, es.T1);
  const int anywide = mg.wide;  // the same in every wave
  if (anywide) {
    __syncthreads();
    for (int64_t i = 0; i < nrec; ++i) {
      if (!(rec[i].wide && !rec[i].bad)) continue;  // uniform: every thread reads the same record
      const int l = (int)(i % L);
      es_moments_tile<double>(pb, (l == 0 ? q1 : q2) + b * V, V, i / L, rec + i, part + i * kEsPart);
      __syncthreads();
    }
    stage(0);
    mg = es_merge<L>(rec, es.T1);
    mg.wide = 1;
  }
  // (2) the plan
  const EsPlan pl = es_make_plan<L>(mg, K);
  if (tid == 0) {
    es.plan[b] = pl;
    if (row_status && pl.flags) row_status[b] |= pl.flags;
  }
  __syncthreads();  // the first chunk and the node ratios are in LDS
  if (pl.nk > 0) {
    // (3) S_l(k), two nodes per thread, tiles in order: nodes up to a tile's kt from
    // its power sums, sum_j (-a_k / a_kt)^j T_j / j!; its window from the stored
    // moments; nothing after the window.  The records and power sums are staged in
    // LDS 64 at a time and the window moments of eight records are loaded at once.
    double S[2][L];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int l = 0; l < L; ++l) S[u][l] = 0.0;
    for (int64_t c0 = 0; c0 < nrec; c0 += kCh) {
      const int nc = (int)min((int64_t)kCh, nrec - c0);
      if (c0 > 0) {
        __syncthreads();  // the previous chunk is consumed
        stage(c0);
        __syncthreads();
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int i = tid + u * kEsThreads;
        if (i >= pl.nk) continue;
        const int k = pl.k_lo + i;
        for (int i0 = 0; i0 < nc; i0 += 8) {
          // eight records at a time, branch-free, so that their LDS reads and window
          // loads are issued together: window starts and lengths (the same in every
          // lane), then each lane's window moment (an in-bounds dummy index when the
          // node is outside the window), then the expansion for the nodes up to kt
          int rkt[8], rnw[8];
          {
            const int4 k0 = *reinterpret_cast<const int4*>(&s_rkt[i0]), k1 = *reinterpret_cast<const int4*>(&s_rkt[i0 + 4]);
            const int4 n0 = *reinterpret_cast<const int4*>(&s_rnw[i0]), n1 = *reinterpret_cast<const int4*>(&s_rnw[i0 + 4]);
            const int kk[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
            const int nn[8] = {n0.x, n0.y, n0.z, n0.w, n1.x, n1.y, n1.z, n1.w};
#pragma unroll
            for (int m = 0; m < 8; ++m) {
              rkt[m] = __builtin_amdgcn_readfirstlane(kk[m]);
              rnw[m] = (i0 + m < nc) ? __builtin_amdgcn_readfirstlane(nn[m]) : -1;  // entries past nc are stale
            }
          }
          double win[8], nx[8];
#pragma unroll
          for (int m = 0; m < 8; ++m) {
            const int ri = min(i0 + m, nc - 1);
            const int d = k - rkt[m];
            const bool in = d >= 1 && d <= rnw[m];
            const double x = part[(c0 + ri) * kEsPart + kEsTaylor + (in ? d - 1 : 0)];
            win[m] = in ? x : 0.0;
            nx[m] = -s_rho[max(0, min(-d, kEsMaxWin - 1))];
          }
#pragma unroll
          for (int m = 0; m < 8; ++m) {
            if (rnw[m] < 0) continue;  // uniform: the record adds nothing
            const int ri = i0 + m;
            double e = s_pow[ri][kEsTaylor - 1];
#pragma unroll
            for (int j = kEsTaylor - 2; j >= 0; --j) e = fma(e, nx[m], s_pow[ri][j]);
            S[u][ri % L] += (k - rkt[m] <= 0) ? e : win[m];  // records are (tile, law) in order; c0 is even
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int i = tid + u * kEsThreads;
      if (i >= pl.nk) continue;
      const int k = pl.k_lo + i;
      const double ha = kEsStep * exp((double)k * kEsStep);
      if (L == 1) {
        const double sm = S[u][0] + (K >= 3 ? pl.q0[0] : 0.0);
        double sp = 1.0;
        for (int j = 1; j < K; ++j) sp *= sm;
        s_c[0][i] = (double)K * ha * sp;
      } else {
        s_c[0][i] = ha * S[u][L - 1];
        s_c[L - 1][i] = ha * S[u][0];
      }
    }
    __syncthreads();
    // the expansion of the grid up to each node: B_j(k) = sum_(k' <= k) c_k' e^(-(k - k') h j), stored / j!
    // The recurrence B_j(k) = rho_j B_j(k - 1) + c_k (rho_j = e^(-jh)) in blocks of 16 nodes: each
    // task (law, j, block) runs it inside its block from zero, then adds the carry of the blocks
    // before it, sum_b' last_b' rho_j^(16 (b - 1 - b')), times rho_j^(m + 1) at offset m.
    if (!pl.fp64) {
      constexpr int kPB = 16;
      const int nblk = (pl.nk + kPB - 1) / kPB;  // <= 30
      const int ntask = L * kEsTaylor * nblk;
      __shared__ double s_last[L][kEsTaylor][(kEsMaxNodes + kPB - 1) / kPB];
      for (int task = tid; task < ntask; task += kEsThreads) {
        const int blk = task % nblk, j = (task / nblk) % kEsTaylor, l = task / (nblk * kEsTaylor);
        const double rho = s_rho[j];
        const int i0 = blk * kPB, n = min(kPB, pl.nk - i0);
        // the block's c loaded first and the recurrence selected, not branched on, per node
        double cv[kPB];
#pragma unroll
        for (int m = 0; m < kPB; ++m) cv[m] = s_c[l][min(i0 + m, kEsMaxWin - 1)];
        double acc = 0.0;
#pragma unroll
        for (int m = 0; m < kPB; ++m) {
          double t = fma(acc, rho, cv[m]);
          __asm__ volatile("" : "+v"(t));
          acc = (m < n) ? t : acc;
        }
        s_last[l][j][blk] = acc;
      }
      __syncthreads();
      for (int task = tid; task < ntask; task += kEsThreads) {
        const int blk = task % nblk, j = (task / nblk) % kEsTaylor, l = task / (nblk * kEsTaylor);
        const double rho = s_rho[j], f = es_inv_fact(j);
        double r16 = rho * rho;  // rho^16
        r16 *= r16;
        r16 *= r16;
        r16 *= r16;
        double carry = 0.0;
        for (int bb = 0; bb < blk; ++bb) carry = fma(carry, r16, s_last[l][j][bb]);
        double* pt = es.ptab + (b * L + l) * (int64_t)kEsMaxNodes * kEsTaylor;
        const int i0 = blk * kPB, n = min(kPB, pl.nk - i0);
        double cv[kPB];
#pragma unroll
        for (int m = 0; m < kPB; ++m) cv[m] = s_c[l][min(i0 + m, kEsMaxWin - 1)];
        double acc = 0.0, pw = rho, out[kPB];
#pragma unroll
        for (int m = 0; m < kPB; ++m) {
          acc = fma(acc, rho, cv[m]);
          out[m] = fma(carry, pw, acc) * f;
          pw *= rho;
        }
#pragma unroll
        for (int m = 0; m < kPB; ++m)
          if (m < n) pt[(i0 + m) * kEsTaylor + j] = out[m];
      }
      // the per-token polynomial of every node row i (k0 = k_lo + i): a query token with
      // x = a_k0 w, t = (x - x_mid) / delta, takes sum_n A_n(i) t^n for its nine node terms
      // and the expansion of the grid below k0,
      //   A_n(i) = sum_m c_(i+m) G[m][n] + sum_j B_j(k0 - 1) / j! H[j][n]
      // (c = 0 off the grid; past the grid's end B_j decays by e^(-jh) per node)
      __syncthreads();  // the prefix table is written
      const int nrow = pl.nrow;  // <= kEsAtabRows
      for (int task = tid; task < L * nrow; task += kEsThreads) {
        const int l = task / nrow, i = task % nrow;
        const double* pt = es.ptab + (b * L + l) * (int64_t)kEsMaxNodes * kEsTaylor;
        double cm[kEsTokNodesC], pj[kEsTaylor], pv[kEsTaylor];
        const int prow = max(0, min(i - 1, pl.nk - 1));  // B_j(k0 - 1): row i - 1, or the last row decayed
        const int past = max(0, i - 1 - prow);              // rows past the grid's end: e^(-jh) a node
        // every load issued unconditionally (clamped indices), then selected
#pragma unroll
        for (int j = 0; j < kEsTaylor; ++j) pv[j] = pt[prow * kEsTaylor + j];
#pragma unroll
        for (int m = 0; m < kEsTokNodesC; ++m) cm[m] = s_c[l][min(i + m, kEsMaxWin - 1)];
#pragma unroll
        for (int m = 0; m < kEsTokNodesC; ++m) cm[m] = (i + m < pl.nk) ? cm[m] : 0.0;
#pragma unroll
        for (int j = 0; j < kEsTaylor; ++j) {
          const double v = (i >= 1) ? pv[j] : 0.0;
          // e^(-past j h) from the table of e^(-mh) (the same expression as its entries);
          // past j beyond the table (weights spanning far beyond the grid) takes exp
          const int m = past * j;
          pj[j] = (m == 0) ? v : v * ((m < kEsMaxWin) ? s_rho[m] : exp(-(double)m * kEsStep));
        }
        double* at = es.atab + ((b * L + l) * (int64_t)kEsAtabRows + i) * kEsPolyLen;
        double a[kEsPolyLen];  // eleven independent sums, interleaved
#pragma unroll
        for (int n = 0; n < kEsPolyLen; ++n) a[n] = 0.0;
#pragma unroll
        for (int m = 0; m < kEsTokNodesC; ++m)
#pragma unroll
          for (int n = 0; n < kEsPolyLen; ++n) a[n] = fma(cm[m], kEsPolyG[m][n], a[n]);
#pragma unroll
        for (int j = 0; j < kEsTaylor; ++j)
#pragma unroll
          for (int n = 0; n < kEsPolyLen; ++n) a[n] = fma(pj[j], kEsPolyH[j][n], a[n]);
#pragma unroll
        for (int n = 0; n < kEsPolyLen; ++n) at[n] = a[n];
      }
    }
  }
  // (4) rows in fp64, from the tables in LDS
  if (pl.fp64) {
    for (int64_t t = 0; t < es.T2; ++t) {
      es_eval_tile<double, L>(pb, q1 + b * V, (L == 2) ? q2 + b * V : nullptr, V, K, t, r + b * V, pl, &s_c[0][0]);
      __syncthreads();
    }
  }
}

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Workgroups of a persistent launch over `tiles` tiles: every resident slot of
// the device once, each workgroup taking the same number of tiles (the last
// ones one fewer).  Occupancy is measured once per device and kernel slot.
constexpr int kEsSlotMoments = 0, kEsSlotEval1 = 1, kEsSlotEval2 = 2, kEsSlots = 3;
template <typename Kern>
static unsigned es_grid(Kern kernel, int64_t tiles, int slot) {
  static int s_slots[64][kEsSlots];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  int slots = s_slots[dev][slot];
  if (slots <= 0) {
    int cus = 0, occ = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, kEsThreads, 0) != hipSuccess) occ = 0;
    slots = std::max(cus, 1) * std::max(occ, 1);
    s_slots[dev][slot] = slots;
  }
  const int64_t per = (tiles + slots - 1) / slots;
  return (unsigned)std::max<int64_t>(1, (tiles + per - 1) / per);
}

void carve_es(void* base, int64_t B, int64_t V, int L, EsWork* es) {
  const int64_t T1 = es_tiles(V, kEsMomTile), T2 = es_tiles(V, kEsEvalTile);
  char* c = static_cast<char*>(base);
  es->tile = reinterpret_cast<EsTile*>(c);
  c += align256(sizeof(EsTile) * B * T1 * L);
  es->part = reinterpret_cast<double*>(c);
  c += align256(sizeof(double) * B * T1 * L * kEsPart);
  es->plan = reinterpret_cast<EsPlan*>(c);
  c += align256(sizeof(EsPlan) * B);
  es->ptab = reinterpret_cast<double*>(c);
  c += align256(sizeof(double) * B * L * kEsMaxNodes * kEsTaylor);
  es->atab = reinterpret_cast<double*>(c);
  es->T1 = T1;
  es->T2 = T2;
  es->T3 = es_tiles(V, kEsTokTile);
}

}  // namespace

size_t workspace_bytes_expsum(int64_t B, int64_t V, int L) {
  const int64_t T1 = es_tiles(V, kEsMomTile);
  return align256(sizeof(EsTile) * B * T1 * L) + align256(sizeof(double) * B * T1 * L * kEsPart) +
         align256(sizeof(EsPlan) * B) + align256(sizeof(double) * B * L * kEsMaxNodes * kEsTaylor) +
         align256(sizeof(double) * B * L * kEsAtabRows * kEsPolyLen);
}

// q2 == nullptr: K i.i.d. drafts from q1; else two draft laws (K = 2).
hipError_t launch_induced_expsum(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, int K,
                                 float* r, int32_t* row_status, void* workspace, hipStream_t st, double* rsum) {
  static_assert(kEsTokTile == kResSub && kEsWaves == kResParts, "one residual sum per wave and evaluation tile");
  const int64_t nsub = (V + kResSub - 1) / kResSub;
  const int L = (q2 != nullptr) ? 2 : 1;
  EsWork es;
  carve_es(workspace, B, V, L, &es);
  const int64_t G1 = B * es.T1 * L, G2 = B * es.T3;
  const unsigned n1 = es_grid(es_moments_kernel, G1, kEsSlotMoments);
  // the summed form (rsum) sets row_status instead of adding to it: cleared here, ahead of the
  // coefficient kernel's flags
  hipLaunchKernelGGL(es_moments_kernel, dim3(n1), dim3(kEsThreads), 0, st, p, q1, q2, V, L, G1,
                     (int)((G1 + n1 - 1) / n1), es, rsum ? row_status : nullptr);
  if (L == 1) {
    hipLaunchKernelGGL((es_coef_kernel<1>), dim3((unsigned)B), dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, es,
                       row_status);
    if (rsum) {  // on the plain variant's grid (its lower occupancy: 1 us faster on 256 x 32000 than its own)
      const unsigned n2 = es_grid(es_eval_kernel<1, false>, G2, kEsSlotEval1);
      hipLaunchKernelGGL((es_eval_kernel<1, true>), dim3(n2), dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, G2,
                         (int)((G2 + n2 - 1) / n2), es, rsum, nsub);
    } else {
      const unsigned n2 = es_grid(es_eval_kernel<1, false>, G2, kEsSlotEval1);
      hipLaunchKernelGGL((es_eval_kernel<1, false>), dim3(n2), dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, G2,
                         (int)((G2 + n2 - 1) / n2), es, rsum, nsub);
    }
  } else {
    hipLaunchKernelGGL((es_coef_kernel<2>), dim3((unsigned)B), dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, es,
                       row_status);
    if (rsum) {
      const unsigned n2 = es_grid(es_eval_kernel<2, false>, G2, kEsSlotEval2);
      hipLaunchKernelGGL((es_eval_kernel<2, true>), dim3(n2), dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, G2,
                         (int)((G2 + n2 - 1) / n2), es, rsum, nsub);
    } else {
      const unsigned n2 = es_grid(es_eval_kernel<2, false>, G2, kEsSlotEval2);
      hipLaunchKernelGGL((es_eval_kernel<2, false>), dim3(n2), dim3(kEsThreads), 0, st, p, q1, q2, V, K, r, G2,
                         (int)((G2 + n2 - 1) / n2), es, rsum, nsub);
    }
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

// ------------------------------------------------------------------ top-s rows
// K i.i.d. drafts from a draft truncated to at most s_max tokens (a top-s draft):
// one workgroup of 1024 threads per row streams p and q once (twice when one wave
// meets more than kTkSeg support tokens), writes r = 0 (the support's entries are
// written again at the end), keeps the support (index, p, q, w) in LDS and takes the
// trapezoidal rule of the tiled path, on the same grid, directly over it:
//   S_k = sum over the support of q(x) exp(-a_k w(x))      (p(x) > 0),
//   r(y) = p(y) sum_k c_k exp(-a_k w(y)),  c_k = K h a_k (S_k [+ Q0 for K >= 3])^(K-1),
// every (node, token) term exactly (no windows, expansions or polynomial tables),
// plus the zero-weight closed forms.  fp32 terms with the tile path's power-of-two
// scale (w' = w 2^tau, rates a_k 2^-tau), fp64 sums of the per-lane partials; a
// row whose weights leave the fp32 normal range, span more than 2^kTkMaxRange or
// need nodes outside the rate table is taken in fp64.
namespace {

constexpr int kTkThreads = 1024;
constexpr int kTkWaves = kTkThreads / 64;
constexpr int kTkCap = MDSS_K3_MAX_SUPPORT;   // support entries held in LDS
constexpr int kTkPer = 4;                     // tokens per thread per streaming step
constexpr int kTkStep = kTkThreads * kTkPer;  // 4096 tokens per step
constexpr int kTkSeg = kTkCap / kTkWaves;     // support tokens of one wave's stream segment
constexpr int kTkLdsParts = 1024;             // residual parts kept in LDS: rows of up to 262144 tokens
constexpr int kTkAhead = 2;                   // streaming steps in flight (64 KB of p and q per workgroup)
constexpr int kTkE = 4;                       // support entries per lane in the node sums
constexpr int kTkGroup = 64 * kTkE;           // entries of one wave group
constexpr int kTkMaxRange = 100;              // binary exponent span of the weights kept in fp32
static_assert(kTkCap % kTkGroup == 0 && kTkCap / kTkGroup <= kTkWaves, "groups of 256 entries, one a wave at most");
static_assert(kTkPer * kTkWaves == 64, "one (slot, wave) count per lane");

// Inclusive scan of an int over the wave: row_shr steps inside each 16-lane row (DPP,
// lanes before a row's start read 0), then the row totals carried by readlane.
__device__ __forceinline__ int tk_scan_int(int v, int lane) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);  // row_shr:8
  const int t0 = __builtin_amdgcn_readlane(v, 15), t1 = __builtin_amdgcn_readlane(v, 31),
            t2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane >> 4;
  return v + (row == 0 ? 0 : (row == 1 ? t0 : (row == 2 ? t0 + t1 : t0 + t1 + t2)));
}

// A streaming step's p and q, thread t holding the four consecutive tokens x0 + 4t ..
// x0 + 4t + 3 (one 16-byte load each when the rows are 16-byte aligned); 0 past the row.
__device__ __forceinline__ void tk_load4(const float* __restrict__ pb, const float* __restrict__ qb, int64_t V,
                                         int64_t x0, int tid, bool vec, float (&pv)[kTkPer], float (&qv)[kTkPer]) {
  static_assert(kTkPer == 4, "one float4 a thread and step");
  const int64_t x = x0 + 4 * tid;
  if (vec && x + 3 < V) {
    const float4 a = *reinterpret_cast<const float4*>(pb + x), c = *reinterpret_cast<const float4*>(qb + x);
    pv[0] = a.x; pv[1] = a.y; pv[2] = a.z; pv[3] = a.w;
    qv[0] = c.x; qv[1] = c.y; qv[2] = c.z; qv[3] = c.w;
  } else {
#pragma unroll
    for (int i = 0; i < kTkPer; ++i) {
      pv[i] = (x + i < V) ? pb[x + i] : 0.0f;
      qv[i] = (x + i < V) ? qb[x + i] : 0.0f;
    }
  }
}

// The token-order pass's step: thread t holding tokens x0 + 1024 i + t (0 past the row's
// end); a whole step without bounds checks.
__device__ __forceinline__ void tk_load(const float* __restrict__ pb, const float* __restrict__ qb, int64_t V,
                                        int64_t x0, int tid, float (&pv)[kTkPer], float (&qv)[kTkPer]) {
  const float* ps = pb + x0 + tid;
  const float* qs = qb + x0 + tid;
  if (x0 + kTkStep <= V) {  // uniform
#pragma unroll
    for (int i = 0; i < kTkPer; ++i) {
      pv[i] = ps[i * kTkThreads];
      qv[i] = qs[i * kTkThreads];
    }
  } else {
    const int rest = (int)(V - x0) - tid;
#pragma unroll
    for (int i = 0; i < kTkPer; ++i) {
      pv[i] = (i * kTkThreads < rest) ? ps[i * kTkThreads] : 0.0f;
      qv[i] = (i * kTkThreads < rest) ? qs[i * kTkThreads] : 0.0f;
    }
  }
}

// kRes: also the residual sums of Algorithm 1 with proposal r (the summed form), one fp64
// sum per 256-token part (rsum[b][part], four parts per 1024-token sub-tile): while the
// row streams, each wave writes the sum of p over its part; once r is written, each
// support token's correction max(0, p - r) - p is added to its part's sum.  row_status is
// set, not OR-ed into.
// kDraw (with kRes): the step in one launch; once r and the sums are complete, wave 0
// takes the row's selection and Algorithm 1 from them (draw_from_sums, the code of
// the summed form's draw), with the drafts, uniforms and outputs of dr.
struct TkDraw {
  const float* u;
  uint64_t seed, offset;
  SelArgs sel;
  int32_t* out_token;
  uint8_t* accepted;
  double* residual_mass;
};
template <bool kRes, bool kDraw>
__global__ __launch_bounds__(kTkThreads) void es_topk_kernel(const float* __restrict__ p, const float* __restrict__ q,
                                                             int64_t V, int K, int s_max, float* __restrict__ r,
                                                             int32_t* __restrict__ row_status,
                                                             double* __restrict__ rsum, int64_t nsub, TkDraw dr) {
  static_assert(kTkStep == 4 * kResSub && kResSub / kResParts == 256 && kTkThreads / 4 == 256,
                "a wave's 256 tokens of a step are one part of the residual sums");
  static_assert(kRes || !kDraw, "the fused draw takes the residual sums");
  __shared__ int s_idx[kTkCap];
  __shared__ float s_p[kTkCap];
  __shared__ float s_q[kTkCap];
  __shared__ float s_w[kTkCap];                    // the weight (unscaled, then w 2^tau in fp32)
  __shared__ float s_part[kTkWaves][kEsMaxNodes];  // per wave: its entries' share of S_k at its nodes
  __shared__ float s_rate[kEsMaxNodes + 16];       // fp32: log2(e) a_k 2^-tau (16 spare entries: 0)
  __shared__ float s_cf[kEsMaxNodes + 16];         // fp32: c_k 2^-tau (0 on the spare entries)
  __shared__ double s_c64[kEsMaxNodes];            // fp64: c_k
  __shared__ int s_cnt[2][64];
  __shared__ int s_flag[kTkWaves];
  __shared__ float s_f[kTkWaves][2];
  __shared__ double s_d[kTkWaves];
  __shared__ double s_e[kTkWaves][2];
  __shared__ int s_n[kTkWaves];
  __shared__ EsPlan s_plan;
  // while streaming: wave w's support tokens (index, p, q) at [w kTkSeg, (w + 1) kTkSeg);
  // once the list is joined, kRes keeps each entry's residual correction here (fp64)
  __shared__ __align__(16) uint32_t s_seg[3 * kTkCap];
  int* const s_sidx = reinterpret_cast<int*>(s_seg);
  float* const s_sp = reinterpret_cast<float*>(s_seg + kTkCap);
  float* const s_sq = reinterpret_cast<float*>(s_seg + 2 * kTkCap);
  double* const s_dres = reinterpret_cast<double*>(s_seg);
  __shared__ int s_wn[kTkWaves];
  // kRes: the parts' sums of a row of up to kTkLdsParts parts are kept here and written
  // out once at the end; longer rows keep them in rsum itself
  __shared__ double s_parts[kRes ? kTkLdsParts : 1];
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t b = blockIdx.x;
  const float* pb = p + b * V;
  const float* qb = q + b * V;
  float* rb = r + b * V;
  if (kRes && tid == 0 && row_status) row_status[b] = 0;  // thread 0 adds the flags below
  const int64_t nparts = nsub * kResParts;
  const bool lds_parts = kRes && nparts <= kTkLdsParts;  // uniform
  double* const parts = lds_parts ? s_parts : rsum + b * nparts;
  // the fused draw, by wave 0 once every thread's r and sums are written (after a barrier);
  // the same 16-byte-load condition as the summed form's draw launch
  const auto draw = [&](const double* sb) {
    if (wid != 0) return;
    const bool dvec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(r)) % 16 == 0);
    if (dvec)
      draw_from_sums<true, true, kResParts, kResSub>(pb, rb, sb, nsub, nullptr, dr.u, dr.seed, dr.offset, b, V, lane,
                                                     dr.out_token, dr.accepted, dr.residual_mass, row_status, dr.sel);
    else
      draw_from_sums<false, true, kResParts, kResSub>(pb, rb, sb, nsub, nullptr, dr.u, dr.seed, dr.offset, b, V, lane,
                                                      dr.out_token, dr.accepted, dr.residual_mass, row_status, dr.sel);
  };

  // (1) stream the row, kTkAhead steps in flight, thread t on the four consecutive tokens
  //     x0 + 4t .. x0 + 4t + 3 of each step (wave w on the 256 tokens x0 + 256w ..): r = 0,
  //     the probability checks, each wave's support tokens appended to its own LDS segment
  //     (no barrier a step), and for kRes each wave's fp64 sum of p over its 256 tokens:
  //     part (x0 >> 8) + w of the residual sums' layout
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(q) |
                                     reinterpret_cast<uintptr_t>(r)) % 16 == 0);
  float pf[kTkAhead][kTkPer], qf[kTkAhead][kTkPer];  // the next kTkAhead steps, in flight
#pragma unroll
  for (int j = 0; j < kTkAhead; ++j) tk_load4(pb, qb, V, (int64_t)j * kTkStep, tid, vec, pf[j], qf[j]);
  int bad = 0, wn = 0;  // wn: this wave's support tokens so far (uniform)
  const int64_t nstep = (V + kTkStep - 1) / kTkStep;
  for (int64_t st = 0; st < nstep; ++st) {
    const int64_t x0 = st * kTkStep;
    float pc[kTkPer], qc[kTkPer];
#pragma unroll
    for (int i = 0; i < kTkPer; ++i) {
      pc[i] = pf[0][i];
      qc[i] = qf[0][i];
#pragma unroll
      for (int j = 0; j + 1 < kTkAhead; ++j) {
        pf[j][i] = pf[j + 1][i];
        qf[j][i] = qf[j + 1][i];
      }
    }
    if (st + kTkAhead < nstep)
      tk_load4(pb, qb, V, x0 + kTkAhead * kTkStep, tid, vec, pf[kTkAhead - 1], qf[kTkAhead - 1]);
    const int64_t x = x0 + 4 * tid;
    // r = 0 over the whole step in full lines (a masked store would leave partial lines);
    // the support's values overwrite these after the sums, past workgroup barriers
    if (vec && x + 3 < V) {
      *reinterpret_cast<float4*>(rb + x) = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    } else {
#pragma unroll
      for (int i = 0; i < kTkPer; ++i)
        if (x + i < V) rb[x + i] = 0.0f;
    }
    if (kRes) {
      double loc = 0.0;
#pragma unroll
      for (int i = 0; i < kTkPer; ++i) loc += (double)pc[i];  // p = 0 past the row's end
      const double tot = wave_sum_dpp(loc);
      const int64_t part = (x0 >> 8) + wid;
      if (lane == 0 && part < nparts) parts[part] = tot;
    }
#pragma unroll
    for (int i = 0; i < kTkPer; ++i) {
      // NaN, -inf, a negative normal or denormal, +inf (-0 is a zero probability)
      bad |= __builtin_amdgcn_classf(pc[i], 0x21F) | __builtin_amdgcn_classf(qc[i], 0x21F);
      const bool sup = qc[i] > 0.0f;  // 0 past the row's end
      const uint64_t mask = __builtin_amdgcn_ballot_w64(sup);
      const int pos = wn + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                          __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
      if (sup && pos < kTkSeg) {
        const int at = wid * kTkSeg + pos;
        s_sidx[at] = (int)x + i;  // rows < 2^31 tokens
        s_sp[at] = pc[i];
        s_sq[at] = qc[i];
      }
      wn += (int)__builtin_popcountll(mask);
    }
  }
  const bool wave_bad = __builtin_amdgcn_ballot_w64(bad != 0) != 0;  // every lane votes
  if (lane == 0) {
    s_flag[wid] = wave_bad ? 1 : 0;
    s_wn[wid] = wn;
  }
  __syncthreads();  // the segments are complete (and a flagged row's NaN below follows its zeros)
  int flags = 0, n = 0, wmax_n = 0, base = 0;
#pragma unroll
  for (int i = 0; i < kTkWaves; ++i) {
    flags |= s_flag[i];
    base += (i < wid) ? s_wn[i] : 0;
    n += s_wn[i];
    wmax_n = max(wmax_n, s_wn[i]);
  }
  flags = flags ? kRowBadProb : (n > s_max ? kRowSupport : 0);
  if (!flags) {  // uniform; here n <= s_max <= kTkCap
    if (wmax_n <= kTkSeg) {
      // (1b) the list: the segments in wave order (each in its tokens' stream order)
      for (int j = lane; j < wn; j += 64) {
        s_idx[base + j] = s_sidx[wid * kTkSeg + j];
        s_p[base + j] = s_sp[wid * kTkSeg + j];
        s_q[base + j] = s_sq[wid * kTkSeg + j];
      }
    } else {
      // (1c) a wave met more than kTkSeg support tokens: the row once more, its support
      //      compacted in token order (token x0 + 1024 i + thread; counts per (slot i,
      //      wave), one scan a step)
#pragma unroll
      for (int j = 0; j < kTkAhead; ++j) tk_load(pb, qb, V, (int64_t)j * kTkStep, tid, pf[j], qf[j]);
      int running = 0;
      for (int64_t st = 0; st < nstep; ++st) {
        const int par = (int)(st & 1);
        const int64_t x0 = st * kTkStep;
        float pc[kTkPer], qc[kTkPer];
#pragma unroll
        for (int i = 0; i < kTkPer; ++i) {
          pc[i] = pf[0][i];
          qc[i] = qf[0][i];
#pragma unroll
          for (int j = 0; j + 1 < kTkAhead; ++j) {
            pf[j][i] = pf[j + 1][i];
            qf[j][i] = qf[j + 1][i];
          }
        }
        if (st + kTkAhead < nstep)
          tk_load(pb, qb, V, x0 + kTkAhead * kTkStep, tid, pf[kTkAhead - 1], qf[kTkAhead - 1]);
        uint64_t mask[kTkPer];
#pragma unroll
        for (int i = 0; i < kTkPer; ++i) {
          mask[i] = __builtin_amdgcn_ballot_w64(qc[i] > 0.0f);
          if (lane == 0) s_cnt[par][i * kTkWaves + wid] = (int)__builtin_popcountll(mask[i]);
        }
        es_lds_barrier();  // (s_cnt by step parity: a step's counts are read before the next barrier)
        const int c = s_cnt[par][lane];
        const int incl = tk_scan_int(c, lane);
        const int ex = incl - c;
        const int xs = (int)x0 + tid;
#pragma unroll
        for (int i = 0; i < kTkPer; ++i) {
          const int pos = running + __builtin_amdgcn_readlane(ex, i * kTkWaves + wid) +
                          (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask[i] >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)mask[i], 0u));
          if (qc[i] > 0.0f && pos < kTkCap) {
            s_idx[pos] = xs + i * kTkThreads;
            s_p[pos] = pc[i];
            s_q[pos] = qc[i];
          }
        }
        running += __builtin_amdgcn_readlane(incl, 63);  // the same in every wave
      }
    }
  }
  __syncthreads();  // the list is complete
  const int nl = min(n, kTkCap);  // entries in LDS (n itself when the row is not flagged)

  // (2) weights and the row's statistics (entry e = thread + 1024 j)
  float wlo = INFINITY, whi = 0.0f;
  double q0 = 0.0;
  int npos = 0;
  for (int e = tid; e < nl; e += kTkThreads) {
    const float pp = s_p[e], qq = s_q[e];
    float w = 0.0f;
    if (pp > 0.0f) {
      w = es_denormal(qq) ? es_ratio_small_q(pp, qq) : es_ratio<float>(pp, qq);
      wlo = fminf(wlo, w);
      whi = fmaxf(whi, w);
      ++npos;
    } else {
      q0 += (double)qq;
    }
    s_w[e] = w;
  }
  wlo = es_wave_ext<false>(wlo);
  whi = es_wave_ext<true>(whi);
  q0 = wave_sum(q0);
  npos = wave_sum_int(npos);
  if (lane == 0) {
    s_f[wid][0] = wlo;
    s_f[wid][1] = whi;
    s_d[wid] = q0;
    s_n[wid] = npos;
  }
  __syncthreads();
  float wmin = s_f[0][0], wmax = s_f[0][1];
  q0 = s_d[0];
  npos = s_n[0];
#pragma unroll
  for (int i = 1; i < kTkWaves; ++i) {
    wmin = fminf(wmin, s_f[i][0]);
    wmax = fmaxf(wmax, s_f[i][1]);
    q0 += s_d[i];
    npos += s_n[i];
  }
  // weights outside the fp32 normal range (a ratio that overflowed or a denormal one):
  // the row's range again in fp64, and the fp64 form below
  const bool wide = !flags && npos > 0 && (!(wmin >= __FLT_MIN__) || !(wmax <= __FLT_MAX__));
  double wmin64 = (double)wmin, wmax64 = (double)wmax;
  if (wide) {  // uniform
    double lo = INFINITY, hi = 0.0;
    for (int e = tid; e < nl; e += kTkThreads) {
      const float pp = s_p[e], qq = s_q[e];
      if (pp > 0.0f) {
        const double w = es_ratio<double>(pp, qq);
        lo = fmin(lo, w);
        hi = fmax(hi, w);
      }
    }
    lo = wave_min64(lo);
    hi = wave_max64(hi);
    if (lane == 0) {
      s_e[wid][0] = lo;
      s_e[wid][1] = hi;
    }
    __syncthreads();
    wmin64 = s_e[0][0];
    wmax64 = s_e[0][1];
#pragma unroll
    for (int i = 1; i < kTkWaves; ++i) {
      wmin64 = fmin(wmin64, s_e[i][0]);
      wmax64 = fmax(wmax64, s_e[i][1]);
    }
  }
  // the grid of the tiled path (same merge statistics, same plan), by wave 0 alone: its
  // fp64 logarithms in every one of the sixteen waves would cost each SIMD four times over
  if (wid == 0) {
    EsMerge m;
    m.wmin[0] = m.wmin[1] = npos > 0 ? wmin64 : INFINITY;
    m.wmax[0] = m.wmax[1] = wmax64;
    m.q0[0] = q0;
    m.q0[1] = 0.0;
    m.npos[0] = npos;
    m.npos[1] = 0;
    m.bad = 0;
    m.wide = 0;
    const EsPlan pw = es_make_plan<1>(m, K);
    if (lane == 0) s_plan = pw;
  }
  __syncthreads();
  const EsPlan pl = s_plan;
  if (!flags) flags = pl.flags;
  if (flags) {  // NaN over the whole row
    if (tid == 0 && row_status) row_status[b] |= flags;
    for (int64_t x = tid; x < V; x += kTkThreads) rb[x] = NAN;
    if (kRes)
      for (int64_t t = tid; t < nparts; t += kTkThreads) rsum[b * nparts + t] = NAN;
  } else {
    const int k_lo = pl.k_lo, nk = pl.nk;
    // fp32 unless a weight is not an fp32 normal (an overflowed or denormal ratio), the
    // weights span more than 2^kTkMaxRange, or a node lies outside the rate table
    bool fp64 = wide;
    int tau = 0, range = 0;
    if (nk > 0 && !fp64) {
      es_scale_f32(wmin, wmax, tau, range);
      fp64 = range > kTkMaxRange || k_lo < kEsNodeLo || k_lo + nk > kEsNodeHi;
    }
    double zw = q0;  // K i.i.d. drafts: Q0^(K-1)
    for (int j = 2; j < K; ++j) zw *= q0;
    if (nk > 0 && !fp64) {
      // (3) fp32: S_k.  Entries in groups of 256 (four a lane); with G groups (a power of
      //     two), wave w takes group w % G and the node blocks of 16 congruent to w / G
      //     modulo 16 / G; each block summed across the wave (reduce-scatter)
      for (int e = tid; e < nl; e += kTkThreads) s_w[e] = ldexpf(s_w[e], tau);
      for (int k = tid; k < nk + 16; k += kTkThreads)  // past the grid: rate 0 (a term of 1, times c = 0)
        s_rate[k] = k < nk ? es_rate_f32(k_lo + k, tau) : 0.0f;
      for (int k = lane; k < nk; k += 64) s_part[wid][k] = 0.0f;
      __syncthreads();
      int G = 1;
      while (G * kTkGroup < nl) G *= 2;  // <= kTkWaves
      const int gi = wid % G, bs = kTkWaves / G;
      float w[kTkE], qq[kTkE];
  #pragma unroll
      for (int e = 0; e < kTkE; ++e) {
        const int x = gi * kTkGroup + e * 64 + lane;  // < kTkCap
        const bool in = x < nl && s_p[x] > 0.0f;
        w[e] = in ? s_w[x] : 0.0f;
        qq[e] = in ? s_q[x] : 0.0f;
      }
      for (int blk = wid / G; blk * 16 < nk; blk += bs)
        es_run_block<16>(w, qq, s_rate + blk * 16, lane, s_part[wid] + blk * 16, min(16, nk - blk * 16));
      __syncthreads();
      // (4) c_k 2^-tau from the fp64 sum of the waves' shares (a wave adds 0 at nodes it does not take)
      for (int k = tid; k < nk; k += kTkThreads) {
        double S = 0.0;
  #pragma unroll
        for (int i = 0; i < kTkWaves; ++i) S += (double)s_part[i][k];  // 0 from the waves that did not take node k
        const double sm = S + (K >= 3 ? q0 : 0.0);
        double sp = 1.0;
        for (int j = 1; j < K; ++j) sp *= sm;
        s_cf[k] = (float)ldexp((double)K * kEsStep * exp((double)(k_lo + k) * kEsStep) * sp, -tau);
      }
      for (int k = nk + tid; k < nk + 16; k += kTkThreads) s_cf[k] = 0.0f;
      __syncthreads();
      // (5) r at the support: every node, blocks of 16 in fp32, the blocks summed in fp64
      for (int e = tid; e < nl; e += kTkThreads) {
        const float pp = s_p[e], qq1 = s_q[e];
        double v;
        if (pp > 0.0f) {
          const float we = s_w[e];
          double acc = 0.0;
          for (int k0 = 0; k0 < nk; k0 += 16) {
            float a = 0.0f;
  #pragma unroll
            for (int i = 0; i < 16; ++i) a = fmaf(s_cf[k0 + i], es_decay(s_rate[k0 + i], we), a);
            acc += (double)a;
          }
          const double quad = ldexp((double)pp * acc, tau);
          v = (K == 2) ? fma(2.0 * (double)qq1, q0, quad) : quad;
        } else {
          v = (double)qq1 * zw;
        }
        rb[s_idx[e]] = (float)v;
        if (kRes) s_dres[e] = residual_of(pp, (float)v) - (double)pp;
      }
    } else if (nk > 0) {
      // (3') fp64: S_k per node (wave w takes the nodes congruent to w), lanes over the entries
      for (int kk = wid; kk < nk; kk += kTkWaves) {
        const double a = exp((double)(k_lo + kk) * kEsStep);
        double acc = 0.0;
        for (int e = lane; e < nl; e += 64) {
          const float pp = s_p[e], qq1 = s_q[e];
          if (pp > 0.0f) acc += (double)qq1 * exp(-a * es_ratio<double>(pp, qq1));
        }
        acc = wave_sum(acc);
        if (lane == 0) {
          const double sm = acc + (K >= 3 ? q0 : 0.0);
          double sp = 1.0;
          for (int j = 1; j < K; ++j) sp *= sm;
          s_c64[kk] = (double)K * kEsStep * a * sp;
        }
      }
      __syncthreads();
      for (int e = tid; e < nl; e += kTkThreads) {
        const float pp = s_p[e], qq1 = s_q[e];
        double v;
        if (pp > 0.0f) {
          const double w = es_ratio<double>(pp, qq1);
          double acc = 0.0;
          for (int kk = 0; kk < nk; ++kk) acc += s_c64[kk] * exp(-exp((double)(k_lo + kk) * kEsStep) * w);
          const double quad = (double)pp * acc;
          v = (K == 2) ? fma(2.0 * (double)qq1, q0, quad) : quad;
        } else {
          v = (double)qq1 * zw;
        }
        rb[s_idx[e]] = (float)v;
        if (kRes) s_dres[e] = residual_of(pp, (float)v) - (double)pp;
      }
    } else {
      // no positive weight: zero-weight tokens only
      for (int e = tid; e < nl; e += kTkThreads) {
        const float v = (float)((double)s_q[e] * zw);
        rb[s_idx[e]] = v;
        if (kRes) s_dres[e] = residual_of(s_p[e], v) - (double)s_p[e];
      }
    }
    if (kRes) {
      // (6) the residual sums: the support entries of one 256-token part are consecutive in
      //     the list (a wave's segment holds its parts in stream order; the token-order list
      //     is sorted); the first entry of each run adds the run's corrections, in list order,
      //     to its part's sum of p
      __syncthreads();  // every correction is in LDS, every part's sum of p written
      for (int e = tid; e < nl; e += kTkThreads) {
        const int key = s_idx[e] >> 8;
        if (e > 0 && (s_idx[e - 1] >> 8) == key) continue;  // not the first entry of its run
        double corr = 0.0;
        for (int f = e; f < nl && (s_idx[f] >> 8) == key; ++f) corr += s_dres[f];
        parts[key] += corr;
      }
      if (lds_parts) {
        __syncthreads();
        for (int64_t t = tid; t < nparts; t += kTkThreads) rsum[b * nparts + t] = s_parts[t];
      }
    }
  }
  if (kDraw) {
    __syncthreads();  // r and the residual sums are complete (a flagged row: NaN sums in rsum)
    draw(flags ? rsum + b * nparts : parts);
  }
}

}  // namespace

hipError_t launch_induced_topk_expsum(const float* p, const float* q, int64_t B, int64_t V, int K, int s_max,
                                      float* r, int32_t* row_status, hipStream_t st, double* rsum) {
  const int64_t nsub = (V + kResSub - 1) / kResSub;
  const TkDraw none = {nullptr, 0, 0, {nullptr, nullptr, nullptr, 0, nullptr, nullptr}, nullptr, nullptr, nullptr};
  if (rsum)
    hipLaunchKernelGGL((es_topk_kernel<true, false>), dim3((unsigned)B), dim3(kTkThreads), 0, st, p, q, V, K, s_max, r,
                       row_status, rsum, nsub, none);
  else
    hipLaunchKernelGGL((es_topk_kernel<false, false>), dim3((unsigned)B), dim3(kTkThreads), 0, st, p, q, V, K, s_max,
                       r, row_status, nullptr, nsub, none);
  return hipGetLastError();
}

hipError_t launch_step_topk_expsum(const float* p, const float* q, const int32_t* drafts, const float* u, uint64_t seed,
                                   uint64_t offset, int64_t B, int64_t V, int K, int s_max, float* r,
                                   int32_t* sel_index, int32_t* sel_token, int32_t* out_token, uint8_t* accepted,
                                   double* residual_mass, int32_t* row_status, double* rsum, hipStream_t st) {
  const int64_t nsub = (V + kResSub - 1) / kResSub;
  const TkDraw dr = {u, seed, offset, {q, nullptr, drafts, K, sel_index, sel_token}, out_token, accepted,
                     residual_mass};
  hipLaunchKernelGGL((es_topk_kernel<true, true>), dim3((unsigned)B), dim3(kTkThreads), 0, st, p, q, V, K, s_max, r,
                     row_status, rsum, nsub, dr);
  return hipGetLastError();
}

// ------------------------------------------------------------------ fixed scratch
// Workspace of the allocation-free variant of the K-draft quadrature: a fixed
// device array, one copy on every GPU the library runs on, held until the
// process ends.  In host code `scratch` names a host-side stand-in, never a
// device address: host code uses only the address hipGetSymbolAddress returns
// for the current device.  Every call on a GPU reuses that GPU's copy (calls
// that overlap on one GPU race on it); the kernels write every scratch entry
// they read, so nothing has to be cleared between calls.
static __device__ __align__(256) unsigned char scratch[MDSS_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};  // per device, set on the first call made on it
}  // namespace

// Device address of the scratch array on the calling thread's current device.
static hipError_t es_scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_induced_expsum_noalloc(const float* p, const float* q, int64_t B, int64_t V, int K, float* r,
                                         int32_t* row_status, hipStream_t st) {
  if (workspace_bytes_expsum(B, V, 1) > (size_t)MDSS_NOALLOC_SCRATCH_BYTES) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = es_scratch_address(&ws);
  if (e != hipSuccess) return e;
  return launch_induced_expsum(p, q, nullptr, B, V, K, r, row_status, ws, st);
}

}  // namespace mdss
