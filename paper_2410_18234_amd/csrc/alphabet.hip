// Truncated alphabet (Section 4, after the truncated linear program), gfx950.
//
// Omega_0 = the m tokens of largest target probability (ties by lower id).  The
// selection and Algorithm 1 run with the renormalised target
// p~ = p 1[Omega_0] / p(Omega_0); their output Z is kept with probability
// p_a = p(Omega_0), otherwise a token is drawn from the complement of Omega_0
// in proportion to p, which gives the target law p overall.
//
// Notation: p = target.
#include "common.h"

#include <math.h>

namespace mdss {

namespace {

constexpr int kAlphaThreads = 1024;
constexpr int kAlphaWaves = kAlphaThreads / 64;

// ascending word = descending p (p >= 0; -0 counts as +0)
__device__ __forceinline__ uint32_t desc_word(float p) { return ~__float_as_uint(p + 0.0f); }

__device__ __forceinline__ int block_exclusive_scan_int(int v, int* red, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int incl = wave_inclusive_scan_int(v, lane);
  if (lane == 63) red[wave] = incl;
  __syncthreads();
  int off = 0, t = 0;
  for (int w = 0; w < kAlphaWaves; ++w) {
    off += w < wave ? red[w] : 0;
    t += red[w];
  }
  __syncthreads();
  *total = t;
  return off + incl - v;
}

__device__ __forceinline__ double block_scan_incl(double v, double* red, double* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const double incl = wave_inclusive_scan(v, lane);
  if (lane == 63) red[wave] = incl;
  __syncthreads();
  double off = 0.0, t = 0.0;
  for (int w = 0; w < kAlphaWaves; ++w) {
    if (w < wave) off += red[w];
    t += red[w];
  }
  __syncthreads();
  *total = t;
  return off + incl;
}

// One workgroup per row: exact rank-m threshold by a 4-digit radix select on
// the words, ties at the threshold resolved by id order, then p~ and p(Omega_0).
__global__ __launch_bounds__(kAlphaThreads) void alphabet_truncate_kernel(const float* __restrict__ p, int64_t V,
                                                                          int m, float* __restrict__ pt,
                                                                          double* __restrict__ mass0,
                                                                          int32_t* __restrict__ row_status) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_prefix, s_k;
  __shared__ int ired[kAlphaWaves];
  __shared__ double dred[kAlphaWaves];
  const int64_t b = blockIdx.x;
  const float* pb = p + b * V;
  float* ptb = pt + b * V;
  const int lane = threadIdx.x & 63;
  // validity
  int bad = 0;
  for (int64_t i = threadIdx.x; i < V; i += kAlphaThreads) bad |= bad_prob(pb[i]) ? 1 : 0;
  bad = __ballot(bad) != 0ull;
  if (lane == 0) ired[threadIdx.x >> 6] = bad;
  __syncthreads();
  int any = 0;
  for (int w = 0; w < kAlphaWaves; ++w) any |= ired[w];
  __syncthreads();
  if (any) {
    for (int64_t i = threadIdx.x; i < V; i += kAlphaThreads) ptb[i] = __int_as_float(0x7fc00000);
    if (threadIdx.x == 0) {
      mass0[b] = __longlong_as_double(0x7ff8000000000000ll);
      if (row_status) row_status[b] |= kRowBadProb;
    }
    return;
  }
  // radix select: the word of rank k = min(m, V) - 1 (0-based) and k's rank among its ties
  if (threadIdx.x == 0) {
    s_prefix = 0u;
    s_k = (uint32_t)(min((int64_t)m, V) - 1);
  }
  uint32_t mask = 0u;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int d = threadIdx.x; d < 256; d += kAlphaThreads) hist[d] = 0u;
    __syncthreads();
    const uint32_t prefix = s_prefix;
    for (int64_t i = threadIdx.x; i < V; i += kAlphaThreads) {
      const uint32_t wd = desc_word(pb[i]);
      if ((wd & mask) == prefix) atomicAdd(&hist[(wd >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      uint32_t c[4], sum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = hist[lane * 4 + j];
        sum += c[j];
      }
      const uint32_t incl = (uint32_t)wave_inclusive_scan_int((int)sum, lane);
      const uint32_t k = s_k;
      uint32_t before = incl - sum;
      // the lane whose range of 4 digits holds rank k picks the digit
      if (before <= k && k < incl) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (k < before + c[j]) {
            s_prefix = prefix | ((uint32_t)(lane * 4 + j) << shift);
            s_k = k - before;
            break;
          }
          before += c[j];
        }
      }
    }
    mask |= 0xffu << shift;
    __syncthreads();
  }
  const uint32_t T = s_prefix;  // threshold word
  const int k_tie = (int)s_k;   // Omega_0 takes the first k_tie + 1 tokens (by id) whose word is T
  // mass of Omega_0, tokens in id order (ties counted by an ordered scan)
  double mass = 0.0;
  int tie_run = 0;
  for (int64_t base = 0; base < V; base += kAlphaThreads) {
    const int64_t i = base + threadIdx.x;
    const uint32_t wd = i < V ? desc_word(pb[i]) : 0xffffffffu;
    const int tie = (i < V && wd == T) ? 1 : 0;
    int tot;
    const int rank = tie_run + block_exclusive_scan_int(tie, ired, &tot);
    tie_run += tot;
    if (i < V && (wd < T || (tie && rank <= k_tie))) mass += (double)pb[i];
  }
  // deterministic block sum
  mass = wave_sum(mass);
  if (lane == 0) dred[threadIdx.x >> 6] = mass;
  __syncthreads();
  double M = 0.0;
  for (int w = 0; w < kAlphaWaves; ++w) M += dred[w];
  __syncthreads();
  tie_run = 0;
  for (int64_t base = 0; base < V; base += kAlphaThreads) {
    const int64_t i = base + threadIdx.x;
    const uint32_t wd = i < V ? desc_word(pb[i]) : 0xffffffffu;
    const int tie = (i < V && wd == T) ? 1 : 0;
    int tot;
    const int rank = tie_run + block_exclusive_scan_int(tie, ired, &tot);
    tie_run += tot;
    if (i < V) {
      const bool in = wd < T || (tie && rank <= k_tie);
      ptb[i] = (in && M > 0.0) ? (float)((double)pb[i] / M) : 0.0f;
    }
  }
  if (threadIdx.x == 0) mass0[b] = M;
}

// Post-processing: keep Z iff u_keep < p_a, else the smallest id j outside
// Omega_0 (p~ = 0) with C_j > u_draw Z_c, C the complement's running p mass.
__global__ __launch_bounds__(kAlphaThreads) void alphabet_post_kernel(
    const float* __restrict__ p, const float* __restrict__ pt, const double* __restrict__ mass0,
    const int32_t* __restrict__ token, const float* __restrict__ u2, uint64_t seed, uint64_t offset, int64_t V,
    int32_t* __restrict__ out_token, uint8_t* __restrict__ kept) {
  __shared__ double dred[kAlphaWaves];
  __shared__ int s_found;
  const int64_t b = blockIdx.x;
  const int32_t z = token[b];
  float uk, ud;
  if (u2) {
    uk = u2[b * 2];
    ud = u2[b * 2 + 1];
  } else {
    const uint64_t pos = offset + (uint64_t)b;
    uint32_t c[4] = {(uint32_t)pos, (uint32_t)(pos >> 32), 0u, 1u};
    philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
    uk = (float)(c[0] >> 8) * 5.9604644775390625e-8f;  // 2^-24
    ud = (float)(c[1] >> 8) * 5.9604644775390625e-8f;
  }
  const double pa = mass0[b];
  if (z < 0 || !((double)uk >= pa)) {  // an invalid Z is passed on; NaN p_a keeps Z
    if (threadIdx.x == 0) {
      out_token[b] = z;
      kept[b] = z >= 0 ? 1 : 0;
    }
    return;
  }
  const float* pb = p + b * V;
  const float* ptb = pt + b * V;
  // complement mass, tiles in id order (the same sums as the draw below)
  double carry = 0.0;
  for (int64_t base = 0; base < V; base += kAlphaThreads) {
    const int64_t i = base + threadIdx.x;
    const double v = (i < V && !(ptb[i] > 0.0f)) ? (double)pb[i] : 0.0;
    double tot;
    block_scan_incl(v, dred, &tot);
    carry += tot;
  }
  const double Zc = carry;
  if (!(Zc > 0.0)) {
    if (threadIdx.x == 0) {
      out_token[b] = z;
      kept[b] = 1;
    }
    return;
  }
  const double t = (double)ud * Zc;
  if (threadIdx.x == 0) s_found = 0x7fffffff;
  __syncthreads();
  carry = 0.0;
  for (int64_t base = 0; base < V; base += kAlphaThreads) {
    const int64_t i = base + threadIdx.x;
    const double v = (i < V && !(ptb[i] > 0.0f)) ? (double)pb[i] : 0.0;
    double tot;
    const double C = carry + block_scan_incl(v, dred, &tot);
    // the draw is the smallest id whose running complement mass exceeds t
    if (i < V && C > t) atomicMin(&s_found, (int)i);
    __syncthreads();
    if (s_found != 0x7fffffff) break;
    carry += tot;
  }
  if (threadIdx.x == 0) {
    const bool drawn = s_found != 0x7fffffff;
    out_token[b] = drawn ? s_found : z;
    kept[b] = drawn ? 0 : 1;
  }
}

}  // namespace

hipError_t launch_alphabet_truncate(const float* p, int64_t B, int64_t V, int m, float* pt, double* mass0,
                                    int32_t* row_status, hipStream_t st) {
  hipLaunchKernelGGL(alphabet_truncate_kernel, dim3((unsigned)B), dim3(kAlphaThreads), 0, st, p, V, m, pt, mass0,
                     row_status);
  return hipGetLastError();
}

hipError_t launch_alphabet_post(const float* p, const float* pt, const double* mass0, const int32_t* token,
                                const float* u2, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                                int32_t* out_token, uint8_t* kept, hipStream_t st) {
  hipLaunchKernelGGL(alphabet_post_kernel, dim3((unsigned)B), dim3(kAlphaThreads), 0, st, p, pt, mass0, token, u2,
                     seed, offset, V, out_token, kept);
  return hipGetLastError();
}

}  // namespace mdss
