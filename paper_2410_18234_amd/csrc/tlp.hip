// Truncated linear program for two drafts (Algorithm 2 with the fixed weights
// of eq. heur and the selected-token distribution of eq. p_Ieq; the sort-free
// variant eq. heur2 / p_Ieq3; the same construction for drafts from two
// different distributions, non-identical appendix), gfx950.
//
// Notation: p = target, q1 / q2 = distributions of the first / second draft
// (q2 = q1 for identical drafts).  Tokens are ranked by the key p - q1 q2
// (fp64, rounded once to fp32; larger first, ties by lower id).  Omega_1 =
// the first s ranked tokens; every pair that touches Omega_2 has a fixed
// winner, only the pairs inside Omega_1 are decided by the linear program.
//
// Per row:
//   rank kernel (one workgroup of 1024 threads):
//     SORTED tail: one stable scatter of the row into 256 bins by the top 8
//       bits of the rank word, each group of bins then sorted in LDS, and one
//       reverse scan over the ranked order: r(k) = q1 q2 + q2(k) S1(k) +
//       q1(k) S2(k) with S_i(k) the q_i mass ranked after k;
//     HALF tail: top-s selection only, then r(k) = q1 q2 + (q2 (A - q1) + q1
//       (B - q2)) / 2 with A, B the Omega_2 masses.
//   LP kernel (one wave): the Omega_1 program maximises sum_k min(p_k, c_k +
//     f_k), where c_k is the fixed part of token k's probability and f_k the
//     share it receives of the Omega_1 pairs' masses m_xy (both drafting
//     orders).  It is solved exactly as a maximum flow: start with every pair
//     credited to its earlier-ranked token, then move mass along shortest
//     augmenting paths (Edmonds-Karp) from tokens above their target mass to
//     tokens below it.  The resulting shares give the selection table w.
#include "common.h"

#include <math.h>

namespace mdss {

namespace {

constexpr int kRankThreads = 1024;
constexpr int kRankWaves = kRankThreads / 64;
constexpr int kMaxS = 16;       // largest s accepted by the library
constexpr int kLpMaxIter = 4096;  // augmentations before a row is flagged (bound for s = 16: (s+2)(s(s-1)+2s) = 4608)
constexpr int kTailSorted = 0;
constexpr int kTailHalf = 1;

struct alignas(16) TlpHdr {
  int32_t s_eff;       // min(s, V)
  int32_t flags;       // row status bits found by the rank kernel
  int32_t pad0, pad1;
  double a_tail;       // q1 mass of Omega_2
  double b_tail;       // q2 mass of Omega_2
  double tail_accept;  // sum over Omega_2 of min(p, r)
  double pad2;
};

// Rank word: ascending order of the word = descending key, so a stable
// ascending sort of (word, id) in id order gives the ranking.
__device__ __forceinline__ uint32_t rank_word(float p, float a, float b) {
  const float key = (float)((double)p - (double)a * (double)b) + 0.0f;  // -0 -> +0
  const uint32_t u = __float_as_uint(key);
  const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}

// Lanes of the wave whose digit equals this lane's (restricted to `act`).
__device__ __forceinline__ uint64_t match_digit(uint32_t d, uint64_t act) {
  uint64_t m = act;
#pragma unroll
  for (int bit = 0; bit < 8; ++bit) {
    const uint64_t bb = __ballot((d >> bit) & 1u);
    m &= ((d >> bit) & 1u) ? bb : ~bb;
  }
  return m;
}

__device__ __forceinline__ uint64_t lanes_below(int lane) { return (1ull << lane) - 1ull; }

// Contiguous segment [lo, hi) of n elements walked by this wave (64 elements
// per step, segments in wave order), so per-wave counting keeps input order.
__device__ __forceinline__ void wave_segment(int n, int* lo, int* hi) {
  const int seg = ((n + kRankWaves - 1) / kRankWaves + 63) & ~63;
  *lo = min(n, (int)(threadIdx.x >> 6) * seg);
  *hi = min(n, *lo + seg);
}

// Per-wave digit counts cnt[w][d] -> output positions: cnt[w][d] = base +
// (elements with a smaller digit) + (elements with digit d in waves < w).
// bin_cnt / bin_start (nullable) receive the digit totals and their starts.
// Returns true if one digit holds all n elements (the pass would not move any).
__device__ __forceinline__ bool digit_offsets(uint32_t (*cnt)[256], uint32_t* tot, uint32_t base, int n,
                                              uint32_t* bin_cnt, uint32_t* bin_start, int* flag) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (threadIdx.x == 0) *flag = 0;
  __syncthreads();
  if (threadIdx.x < 256) {
    const int d = threadIdx.x;
    uint32_t run = 0;
    for (int w = 0; w < kRankWaves; ++w) {
      const uint32_t c = cnt[w][d];
      cnt[w][d] = run;
      run += c;
    }
    tot[d] = run;
    if (bin_cnt) bin_cnt[d] = run;
    if (run == (uint32_t)n) *flag = 1;
  }
  __syncthreads();
  if (wave == 0) {
    uint32_t v[4];
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = tot[lane * 4 + j];
      sum += v[j];
    }
    const int incl = wave_inclusive_scan_int((int)sum, lane);
    uint32_t run = base + (uint32_t)incl - sum;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      tot[lane * 4 + j] = run;
      if (bin_start) bin_start[lane * 4 + j] = run;
      run += v[j];
    }
  }
  __syncthreads();
  if (threadIdx.x < 256) {
    const int d = threadIdx.x;
    const uint32_t b0 = tot[d];
    for (int w = 0; w < kRankWaves; ++w) cnt[w][d] += b0;
  }
  const bool uniform = *flag != 0;
  __syncthreads();
  return uniform;
}

// One stable counting pass on bits [shift, shift + 8) of the words,
// (kin, iin) -> (kout, iout), over n elements (global memory or LDS).
// Returns false, writing nothing, when every element has the same digit.
__device__ __forceinline__ bool radix_pass(const uint32_t* kin, const uint32_t* iin, uint32_t* kout, uint32_t* iout,
                                           int n, int shift, uint32_t (*cnt)[256], uint32_t* tot, int* flag) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int lo, hi;
  wave_segment(n, &lo, &hi);
  for (int d = lane; d < 256; d += 64) cnt[wave][d] = 0u;
  constexpr int kBatch = 8;
  for (int base = lo; base < hi; base += 64 * kBatch) {
    uint32_t kr[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      kr[j] = i < hi ? kin[i] : 0u;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      const uint64_t act = __ballot(i < hi);
      if (!act) break;
      const uint32_t d = (kr[j] >> shift) & 255u;
      const uint64_t m = match_digit(d, act);
      if (i < hi && lane == __ffsll((long long)m) - 1) cnt[wave][d] += (uint32_t)__popcll(m);
    }
  }
  __syncthreads();
  if (digit_offsets(cnt, tot, 0u, n, nullptr, nullptr, flag)) return false;
  for (int base = lo; base < hi; base += 64 * kBatch) {
    uint32_t kr[kBatch], ir[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      kr[j] = i < hi ? kin[i] : 0u;
      ir[j] = i < hi ? iin[i] : 0u;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      const uint64_t act = __ballot(i < hi);
      if (!act) break;
      const uint32_t d = (kr[j] >> shift) & 255u;
      const uint64_t m = match_digit(d, act);
      if (i < hi) {
        const uint32_t pos = cnt[wave][d] + (uint32_t)__popcll(m & lanes_below(lane));
        kout[pos] = kr[j];
        iout[pos] = ir[j];
        if (lane == __ffsll((long long)m) - 1) cnt[wave][d] += (uint32_t)__popcll(m);
      }
    }
  }
  __syncthreads();
  return true;
}

__device__ __forceinline__ void flag_row(int64_t b, int64_t V, int s, float* rb, int32_t* omega1, TlpHdr* hdr,
                         int32_t* row_status, int flags) {
  for (int64_t i = threadIdx.x; i < V; i += kRankThreads) rb[i] = __int_as_float(0x7fc00000);
  if (threadIdx.x < s) omega1[b * s + threadIdx.x] = -1;
  if (threadIdx.x == 0) {
    TlpHdr h = {};
    h.flags = flags;
    hdr[b] = h;
    if (row_status) row_status[b] |= flags;
  }
}

// Block-wide sum in a fixed order (wave tree, then waves in index order).
__device__ __forceinline__ double block_sum(double v, double* red) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double t = 0.0;
  for (int w = 0; w < kRankWaves; ++w) t += red[w];
  __syncthreads();
  return t;
}

// Exclusive suffix sums over the block in thread order (the sum over higher
// threads), two values at once; also returns the block totals.
__device__ __forceinline__ void block_exclusive_suffix2(double a, double b, double* ea, double* eb, double* ta,
                                                        double* tb, double* sa, double* sb) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  double ia = a, ib = b;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double oa = __shfl_down(ia, off, 64), ob = __shfl_down(ib, off, 64);
    if (lane + off < 64) {
      ia += oa;
      ib += ob;
    }
  }
  double xa = __shfl_down(ia, 1, 64), xb = __shfl_down(ib, 1, 64);
  if (lane == 63) xa = xb = 0.0;
  if (lane == 0) {
    sa[wave] = ia;
    sb[wave] = ib;
  }
  __syncthreads();
  double oa = 0.0, ob = 0.0, fa = 0.0, fb = 0.0;
  for (int w = kRankWaves - 1; w >= 0; --w) {
    if (w > wave) {
      oa += sa[w];
      ob += sb[w];
    }
    fa += sa[w];
    fb += sb[w];
  }
  __syncthreads();
  *ea = oa + xa;
  *eb = ob + xb;
  *ta = fa;
  *tb = fb;
}

// ---------------------------------------------------------------- SORTED tail
// Bin-ordered copy of a row made by the scatter pass (structure of arrays).
struct BinRow {
  uint32_t* word;
  uint32_t* id;
  float* p;
  float* a;
  float* b;
};

constexpr int kGroup = 8192;  // entries sorted in LDS at once

// Reverse scan of one ranked chunk: sorted[g] (g < G <= kGroup) = index into
// the bin order of the entry with rank first_rank + g.  Entries ranked in
// Omega_1 are recorded and take no part in the sums; every other entry k gets
// r(k) = a b + b S_a + a S_b with S the q1 / q2 mass ranked after k.
// The entries are first gathered (thread-strided, many loads in flight) into
// the LDS staging arrays A, Bq, P, ID (kGroup entries each; `sorted` may
// alias one of them), then scanned from LDS, E consecutive ranks per thread.
constexpr int kStride = kGroup / kRankThreads;
__device__ __forceinline__ void scan_chunk(const uint32_t* sorted, int G, uint32_t first_rank, uint32_t bin_base,
                                           const BinRow& br, int s, int64_t b, float* rb, int32_t* omega1,
                                           double* ca, double* cb, double* acc, double* sa, double* sb, float* A,
                                           float* Bq, float* P, uint32_t* ID) {
  uint32_t at[kStride];
#pragma unroll
  for (int k = 0; k < kStride; ++k) {
    const int g = (int)threadIdx.x + k * kRankThreads;
    at[k] = g < G ? bin_base + sorted[g] : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kStride; ++k) {
    const int g = (int)threadIdx.x + k * kRankThreads;
    if (g < G) {
      A[g] = br.a[at[k]];
      Bq[g] = br.b[at[k]];
      P[g] = br.p[at[k]];
      ID[g] = br.id[at[k]];
    }
  }
  __syncthreads();
  const int E = (G + kRankThreads - 1) / kRankThreads;
  const int g0 = min(G, (int)threadIdx.x * E), g1 = min(G, g0 + E);
  double la = 0.0, lb = 0.0;  // this thread's Omega_2 mass (consecutive ranks)
  for (int g = g0; g < g1; ++g) {
    if (first_rank + (uint32_t)g < (uint32_t)s) continue;
    la += (double)A[g];
    lb += (double)Bq[g];
  }
  double ea, eb, ta, tb;
  block_exclusive_suffix2(la, lb, &ea, &eb, &ta, &tb, sa, sb);
  double s1 = *ca + ea, s2 = *cb + eb;  // mass ranked after the entry being visited
  for (int g = g1 - 1; g >= g0; --g) {
    const uint32_t rank = first_rank + (uint32_t)g;
    const int id = (int)ID[g];
    if (rank < (uint32_t)s) {
      omega1[b * s + rank] = id;
      continue;
    }
    const double av = (double)A[g], bv = (double)Bq[g];
    const double rv = av * bv + bv * s1 + av * s2;
    rb[id] = (float)rv;
    *acc += fmin((double)P[g], rv);
    s1 += av;
    s2 += bv;
  }
  *ca += ta;
  *cb += tb;
  __syncthreads();  // the staging arrays are reused by the next chunk
}

// One workgroup per row.  Pass 1 counts the top 8 bits of the rank words per
// wave (stable) and checks the row; pass 2 scatters (word, id, p, q1, q2) into
// bin order; then bins are taken from the last-ranked down, consecutive bins
// grouped up to kGroup entries, each group sorted in LDS (stable LSD passes) and
// scanned.  A single bin above kGroup entries is sorted by global LSD passes on
// its lower 24 bits and scanned in chunks.
__global__ __launch_bounds__(kRankThreads) void tlp_rank_sorted_kernel(
    const float* __restrict__ p, const float* __restrict__ q1, const float* __restrict__ q2, int64_t V, int s,
    float* __restrict__ r, int32_t* __restrict__ omega1, TlpHdr* __restrict__ hdr, BinRow bins,
    uint32_t* __restrict__ kA, uint32_t* __restrict__ iA, uint32_t* __restrict__ kB, uint32_t* __restrict__ iB,
    int32_t* __restrict__ row_status) {
  __shared__ uint32_t cnt[kRankWaves][256];
  __shared__ uint32_t tot[256], bin_cnt[256], bin_start[256];
  __shared__ uint32_t kx[2][kGroup], ix[2][kGroup];
  __shared__ double sa[kRankWaves], sb[kRankWaves];
  __shared__ int red[kRankWaves];
  __shared__ int flag;
  const int64_t b = blockIdx.x;
  const float* pb = p + b * V;
  const float* ab = q1 + b * V;
  const float* bb = q2 + b * V;
  float* rb = r + b * V;
  const int n = (int)V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const BinRow br = {bins.word + b * V, bins.id + b * V, bins.p + b * V, bins.a + b * V, bins.b + b * V};
  int lo, hi;
  wave_segment(n, &lo, &hi);
  constexpr int kBatch = 4;
  // pass 1: validity and per-wave counts of the top digit
  for (int d = lane; d < 256; d += 64) cnt[wave][d] = 0u;
  int bad = 0;
  for (int base = lo; base < hi; base += 64 * kBatch) {
    float pr[kBatch], ar[kBatch], brr[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      pr[j] = i < hi ? pb[i] : 0.0f;
      ar[j] = i < hi ? ab[i] : 0.0f;
      brr[j] = i < hi ? bb[i] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      const uint64_t act = __ballot(i < hi);
      if (!act) break;
      bad |= (bad_prob(pr[j]) || bad_prob(ar[j]) || bad_prob(brr[j])) ? 1 : 0;
      const uint32_t d = rank_word(pr[j], ar[j], brr[j]) >> 24;
      const uint64_t m = match_digit(d, act);
      if (i < hi && lane == __ffsll((long long)m) - 1) cnt[wave][d] += (uint32_t)__popcll(m);
    }
  }
  bad = __ballot(bad) != 0ull;
  if (lane == 0) red[wave] = bad;
  __syncthreads();
  int any = 0;
  for (int w = 0; w < kRankWaves; ++w) any |= red[w];
  if (any) {
    flag_row(b, V, s, rb, omega1, hdr, row_status, kRowBadProb);
    return;
  }
  digit_offsets(cnt, tot, 0u, n, bin_cnt, bin_start, &flag);
  // pass 2: stable scatter into bin order, with the values the scan needs
  for (int base = lo; base < hi; base += 64 * kBatch) {
    float pr[kBatch], ar[kBatch], brr[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      pr[j] = i < hi ? pb[i] : 0.0f;
      ar[j] = i < hi ? ab[i] : 0.0f;
      brr[j] = i < hi ? bb[i] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      const uint64_t act = __ballot(i < hi);
      if (!act) break;
      const uint32_t wd = rank_word(pr[j], ar[j], brr[j]);
      const uint32_t d = wd >> 24;
      const uint64_t m = match_digit(d, act);
      if (i < hi) {
        const uint32_t pos = cnt[wave][d] + (uint32_t)__popcll(m & lanes_below(lane));
        br.word[pos] = wd;
        br.id[pos] = (uint32_t)i;
        br.p[pos] = pr[j];
        br.a[pos] = ar[j];
        br.b[pos] = brr[j];
        if (lane == __ffsll((long long)m) - 1) cnt[wave][d] += (uint32_t)__popcll(m);
      }
    }
  }
  __syncthreads();
  // pass 3: groups of bins, last-ranked first
  double ca = 0.0, cb = 0.0, acc = 0.0;
  int dh = 255;
  while (dh >= 0) {
    int dl = dh;
    uint32_t G = bin_cnt[dh];
    while (dl > 0 && G + bin_cnt[dl - 1] <= (uint32_t)kGroup) G += bin_cnt[--dl];
    const uint32_t g_lo = bin_start[dl];
    if (G == 0) {
      dh = dl - 1;
      continue;
    }
    if (G <= (uint32_t)kGroup) {
      for (uint32_t g = threadIdx.x; g < G; g += kRankThreads) {
        kx[0][g] = br.word[g_lo + g];
        ix[0][g] = g;
      }
      __syncthreads();
      int nonempty = 0;
      for (int d = dl; d <= dh; ++d) nonempty += bin_cnt[d] > 0u;
      const int top = nonempty > 1 ? 32 : 24;  // one bin: the top digit is shared
      int cur = 0;
      for (int shift = 0; shift < top; shift += 8)
        if (radix_pass(kx[cur], ix[cur], kx[cur ^ 1], ix[cur ^ 1], (int)G, shift, cnt, tot, &flag)) cur ^= 1;
      scan_chunk(ix[cur], (int)G, g_lo, g_lo, br, s, b, rb, omega1, &ca, &cb, &acc, sa, sb,
                 reinterpret_cast<float*>(kx[0]), reinterpret_cast<float*>(kx[1]), reinterpret_cast<float*>(ix[0]),
                 ix[1]);
    } else {
      // one bin above the LDS capacity: its words share the top digit
      uint32_t* ka = kA + b * V;
      uint32_t* ia = iA + b * V;
      uint32_t* kb = kB + b * V;
      uint32_t* ib = iB + b * V;
      for (uint32_t g = threadIdx.x; g < G; g += kRankThreads) {
        ka[g] = br.word[g_lo + g];
        ia[g] = g;
      }
      __syncthreads();
      uint32_t *k_in = ka, *i_in = ia, *k_out = kb, *i_out = ib;
      for (int shift = 0; shift < 24; shift += 8) {
        if (radix_pass(k_in, i_in, k_out, i_out, (int)G, shift, cnt, tot, &flag)) {
          uint32_t* t = k_in;
          k_in = k_out;
          k_out = t;
          t = i_in;
          i_in = i_out;
          i_out = t;
        }
      }
      const uint32_t* sorted = i_in;
      const int chunks = (int)((G + kGroup - 1) / kGroup);
      for (int c = chunks - 1; c >= 0; --c) {
        const uint32_t c0 = (uint32_t)c * kGroup;
        const int Gc = (int)min((uint32_t)kGroup, G - c0);
        scan_chunk(sorted + c0, Gc, g_lo + c0, g_lo, br, s, b, rb, omega1, &ca, &cb, &acc, sa, sb,
                   reinterpret_cast<float*>(kx[0]), reinterpret_cast<float*>(kx[1]),
                   reinterpret_cast<float*>(ix[0]), ix[1]);
      }
    }
    dh = dl - 1;
  }
  const int se = min(s, n);
  if (threadIdx.x >= se && threadIdx.x < s) omega1[b * s + threadIdx.x] = -1;
  acc = block_sum(acc, sa);
  if (threadIdx.x == 0) {
    TlpHdr h = {};
    h.s_eff = se;
    h.a_tail = ca;
    h.b_tail = cb;
    h.tail_accept = acc;
    hdr[b] = h;
  }
}

// ------------------------------------------------------------------ HALF tail
// Composite rank: (rank word, id); the smallest composites are the first ranked.
__device__ __forceinline__ uint64_t composite(float p, float a, float b, int id) {
  return ((uint64_t)rank_word(p, a, b) << 32) | (uint32_t)id;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off, 64);
    v = o < v ? o : v;
  }
  return v;
}

// Pop the smallest head among the lanes' sorted lists `l` (ascending), `rounds`
// times; returns the popped values in order in out[0..rounds) (all lanes).
__device__ __forceinline__ void wave_merge_smallest(uint64_t (&l)[kMaxS], int rounds, uint64_t (&out)[kMaxS]) {
#pragma unroll
  for (int t = 0; t < kMaxS; ++t) {
    if (t >= rounds) break;
    const uint64_t m = wave_min_u64(l[0]);
    out[t] = m;
    if (l[0] == m) {  // composites are unique; the padding value never reaches a real round
#pragma unroll
      for (int j = 0; j < kMaxS - 1; ++j) l[j] = l[j + 1];
      l[kMaxS - 1] = ~0ull;
    }
  }
}

__global__ __launch_bounds__(kRankThreads) void tlp_rank_half_kernel(
    const float* __restrict__ p, const float* __restrict__ q1, const float* __restrict__ q2, int64_t V, int s,
    float* __restrict__ r, int32_t* __restrict__ omega1, TlpHdr* __restrict__ hdr,
    int32_t* __restrict__ row_status) {
  __shared__ uint64_t wbest[kRankWaves][kMaxS];
  __shared__ uint64_t best[kMaxS];
  __shared__ double sa[kRankWaves];
  __shared__ int red[kRankWaves];
  const int64_t b = blockIdx.x;
  const float* pb = p + b * V;
  const float* ab = q1 + b * V;
  const float* bb = q2 + b * V;
  float* rb = r + b * V;
  const int n = (int)V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int se = min(s, n);
  // pass 1: validity and the s smallest composites per thread (sorted), then per wave, then per block
  uint64_t l[kMaxS];
#pragma unroll
  for (int j = 0; j < kMaxS; ++j) l[j] = ~0ull;
  int bad = 0;
  for (int i = threadIdx.x; i < n; i += kRankThreads) {
    const float pv = pb[i], av = ab[i], bv = bb[i];
    bad |= (bad_prob(pv) || bad_prob(av) || bad_prob(bv)) ? 1 : 0;
    const uint64_t c = composite(pv, av, bv, i);
    if (c < l[kMaxS - 1]) {
#pragma unroll
      for (int j = kMaxS - 1; j > 0; --j) {
        const uint64_t hi = l[j - 1] > c ? l[j - 1] : c;
        l[j] = l[j] < hi ? l[j] : hi;
      }
      l[0] = l[0] < c ? l[0] : c;
    }
  }
  bad = __ballot(bad) != 0ull;
  if (lane == 0) red[wave] = bad;
  __syncthreads();
  int any = 0;
  for (int w = 0; w < kRankWaves; ++w) any |= red[w];
  if (any) {
    flag_row(b, V, s, rb, omega1, hdr, row_status, kRowBadProb);
    return;
  }
  uint64_t got[kMaxS];
  wave_merge_smallest(l, se, got);
  if (lane == 0) {
#pragma unroll
    for (int t = 0; t < kMaxS; ++t) wbest[wave][t] = t < se ? got[t] : ~0ull;
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int j = 0; j < kMaxS; ++j) l[j] = lane < kRankWaves ? wbest[lane][j] : ~0ull;
    wave_merge_smallest(l, se, got);
    if (lane == 0) {
#pragma unroll
      for (int t = 0; t < kMaxS; ++t) best[t] = t < se ? got[t] : ~0ull;
    }
  }
  __syncthreads();
  if (threadIdx.x < s) omega1[b * s + threadIdx.x] = threadIdx.x < se ? (int32_t)(uint32_t)best[threadIdx.x] : -1;
  int om[kMaxS];  // Omega_1 ids (-1 past s_eff)
#pragma unroll
  for (int t = 0; t < kMaxS; ++t) om[t] = t < se ? (int)(uint32_t)best[t] : -1;
  auto in_omega1 = [&](int i) {
    bool hit = false;
#pragma unroll
    for (int t = 0; t < kMaxS; ++t) hit |= om[t] == i;
    return hit;
  };
  // pass 2: Omega_2 masses
  double A = 0.0, Bm = 0.0;
  for (int i = threadIdx.x; i < n; i += kRankThreads) {
    const float av = ab[i], bv = bb[i];
    if (in_omega1(i)) continue;
    A += (double)av;
    Bm += (double)bv;
  }
  A = block_sum(A, sa);
  Bm = block_sum(Bm, sa);
  // pass 3: r(k) = q1 q2 + (q2 (A - q1) + q1 (B - q2)) / 2 = (q2 A + q1 B) / 2 on Omega_2
  double acc = 0.0;
  for (int i = threadIdx.x; i < n; i += kRankThreads) {
    const float av = ab[i], bv = bb[i], pv = pb[i];
    if (in_omega1(i)) continue;
    const double rv = 0.5 * ((double)bv * A + (double)av * Bm);
    rb[i] = (float)rv;
    acc += fmin((double)pv, rv);
  }
  acc = block_sum(acc, sa);
  if (threadIdx.x == 0) {
    TlpHdr h = {};
    h.s_eff = se;
    h.a_tail = A;
    h.b_tail = Bm;
    h.tail_accept = acc;
    hdr[b] = h;
  }
}

// ------------------------------------------------------------------------ LP
__device__ __forceinline__ double pick(const double (&v)[kMaxS], int j) {
  double t = 0.0;
#pragma unroll
  for (int k = 0; k < kMaxS; ++k)
    if (k == j) t = v[k];
  return t;
}
__device__ __forceinline__ void add_at(double (&v)[kMaxS], int j, double d) {
#pragma unroll
  for (int k = 0; k < kMaxS; ++k)
    if (k == j) v[k] += d;
}

// One wave per row; lane x < s_eff holds Omega_1 token x.  Lane y keeps column
// y of the allocation: col[x] = share of pair {x, y} currently credited to x.
__global__ __launch_bounds__(64) void tlp_lp_kernel(const float* __restrict__ p, const float* __restrict__ q1,
                                                    const float* __restrict__ q2, int64_t V, int s,
                                                    const TlpHdr* __restrict__ hdr, const int32_t* __restrict__ omega1,
                                                    float* __restrict__ r, double* __restrict__ w,
                                                    double* __restrict__ accept, int32_t* __restrict__ row_status) {
  __shared__ double W[kMaxS][kMaxS];
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  const TlpHdr h = hdr[b];
  double* wb = w + b * (int64_t)s * s;
  if (h.flags) {
    for (int i = lane; i < s * s; i += 64) wb[i] = __longlong_as_double(0x7ff8000000000000ll);
    if (lane == 0 && accept) accept[b] = __longlong_as_double(0x7ff8000000000000ll);
    return;
  }
  const int se = h.s_eff;
  const bool mine = lane < se;
  int id = 0;
  double px = 0.0, ax = 0.0, bx = 0.0;
  if (mine) {
    id = omega1[b * s + lane];
    px = (double)p[b * V + id];
    ax = (double)q1[b * V + id];
    bx = (double)q2[b * V + id];
  }
  const double c = ax * bx + bx * h.a_tail + ax * h.b_tail;
  double mc[kMaxS], col[kMaxS];
  double load = c;
#pragma unroll
  for (int v = 0; v < kMaxS; ++v) {
    const double av = __shfl(ax, v, 64), bv = __shfl(bx, v, 64);
    mc[v] = (mine && v < se && v != lane) ? av * bx + ax * bv : 0.0;  // m[v][lane] = m[lane][v]
    col[v] = v < lane ? mc[v] : 0.0;                                    // earlier-ranked token first
    if (v > lane) load += mc[v];
  }
  double ex = mine ? load - px : 0.0;
  bool capped = false;
  for (int iter = 0;; ++iter) {
    const uint64_t src = __ballot(mine && ex > 0.0);
    const uint64_t dst = __ballot(mine && ex < 0.0);
    if (!src || !dst) break;
    if (iter >= kLpMaxIter) {
      capped = true;
      break;
    }
    // breadth-first search from every surplus token over edges x -> y with col_y[x] > 0
    int parent = -1;
    uint64_t visited = src, frontier = src;
    int found = -1;
    while (frontier) {
      bool got = false;
      if (mine && !((visited >> lane) & 1ull)) {
#pragma unroll
        for (int v = 0; v < kMaxS; ++v)
          if (!got && ((frontier >> v) & 1ull) && col[v] > 0.0) {
            parent = v;
            got = true;
          }
      }
      const uint64_t nf = __ballot(got);
      visited |= nf;
      const uint64_t hit = nf & dst;
      if (hit) {
        found = __ffsll((long long)hit) - 1;
        break;
      }
      frontier = nf;
    }
    if (found < 0) break;
    double delta = -__shfl(ex, found, 64);
    int u = found;
    for (int step = 0; step < kMaxS; ++step) {
      const int v = __shfl(parent, u, 64);
      if (v < 0) break;
      delta = fmin(delta, __shfl(pick(col, v), u, 64));
      u = v;
    }
    const int source = u;
    delta = fmin(delta, __shfl(ex, source, 64));
    u = found;
    for (int step = 0; step < kMaxS; ++step) {
      const int v = __shfl(parent, u, 64);
      if (v < 0) break;
      if (lane == u) add_at(col, v, -delta);
      if (lane == v) add_at(col, u, delta);
      u = v;
    }
    if (lane == source) ex -= delta;
    if (lane == found) ex += delta;
  }
  // selection table: W[x][y] = Pr(Y = x | drafted pair {x, y}), either order
  if (mine) {
#pragma unroll
    for (int x = 0; x < kMaxS; ++x) {
      if (x < lane) {
        double wv = mc[x] > 0.0 ? col[x] / mc[x] : 1.0;
        wv = fmin(1.0, fmax(0.0, wv));
        W[x][lane] = wv;
        W[lane][x] = 1.0 - wv;
      }
    }
    W[lane][lane] = 1.0;
  }
  __syncthreads();
  for (int i = lane; i < s * s; i += 64) {
    const int x = i / s, y = i % s;
    wb[i] = (x < se && y < se) ? W[x][y] : 0.0;
  }
  double rv = c;
  if (mine) {
#pragma unroll
    for (int y = 0; y < kMaxS; ++y)
      if (y < se && y != lane) rv += mc[y] * W[lane][y];
    r[b * V + id] = (float)rv;
  }
  const double obj = wave_sum(mine ? fmin(px, rv) : 0.0);
  if (lane == 0) {
    if (accept) accept[b] = h.tail_accept + obj;
    if (capped && row_status) row_status[b] |= kRowLpLimit;
  }
}

// ------------------------------------------------------------------ selection
__global__ __launch_bounds__(256) void tlp_select_kernel(
    const float* __restrict__ p, const float* __restrict__ q1, const float* __restrict__ q2,
    const int32_t* __restrict__ drafts, const float* __restrict__ u, uint64_t seed, uint64_t offset, int64_t B,
    int64_t V, int s, int tail, const int32_t* __restrict__ omega1, const double* __restrict__ w,
    int32_t* __restrict__ sel_index, int32_t* __restrict__ sel_token, int32_t* __restrict__ row_status) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int32_t x1 = drafts[b * 2], x2 = drafts[b * 2 + 1];
  int st = 0;
  if (omega1[b * s] < 0) {
    st = kRowBadProb;  // the plan flagged this row
  } else if (x1 < 0 || (int64_t)x1 >= V || x2 < 0 || (int64_t)x2 >= V) {
    st = kRowBadDraft;
  } else if (!(q1[b * V + x1] > 0.0f) || !(q2[b * V + x2] > 0.0f)) {
    st = kRowBadDraft;
  }
  if (st) {
    sel_index[b] = -1;
    sel_token[b] = -1;
    if (row_status) row_status[b] |= st;
    return;
  }
  float uu[3];
  position_uniforms(u, seed, offset, b, uu);
  int idx = 0;
  if (x1 != x2) {
    int i1 = -1, i2 = -1;
    for (int t = 0; t < s; ++t) {
      const int32_t o = omega1[b * s + t];
      if (o == x1) i1 = t;
      if (o == x2) i2 = t;
    }
    double f;
    if (i1 >= 0 && i2 >= 0) {
      const double* wb = w + b * (int64_t)s * s;
      f = i1 < i2 ? wb[i1 * s + i2] : 1.0 - wb[i2 * s + i1];
    } else if (i1 >= 0) {
      f = 1.0;
    } else if (i2 >= 0) {
      f = 0.0;
    } else if (tail == kTailHalf) {
      f = 0.5;
    } else {
      const uint32_t k1 = rank_word(p[b * V + x1], q1[b * V + x1], q2[b * V + x1]);
      const uint32_t k2 = rank_word(p[b * V + x2], q1[b * V + x2], q2[b * V + x2]);
      f = (k1 < k2 || (k1 == k2 && x1 < x2)) ? 1.0 : 0.0;
    }
    idx = (double)uu[0] < f ? 0 : 1;
  }
  sel_index[b] = idx;
  sel_token[b] = idx == 0 ? x1 : x2;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

// SORTED tail: 5 planes of the bin-ordered row copy + 4 planes for a bin
// above the LDS capacity, each [B][V] 32-bit words.
size_t workspace_bytes_tlp(int64_t B, int64_t V, int tail) {
  size_t bytes = align256((size_t)B * sizeof(TlpHdr));
  if (tail == kTailSorted) bytes += 9 * align256((size_t)B * (size_t)V * sizeof(uint32_t));
  return bytes;
}

hipError_t launch_tlp(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, int s, int tail,
                      float* r, int32_t* omega1, double* w, double* accept, int32_t* row_status, void* workspace,
                      hipStream_t st) {
  if (!q2) q2 = q1;
  char* base = static_cast<char*>(workspace);
  TlpHdr* hdr = reinterpret_cast<TlpHdr*>(base);
  base += align256((size_t)B * sizeof(TlpHdr));
  if (tail == kTailSorted) {
    const size_t plane = align256((size_t)B * (size_t)V * sizeof(uint32_t));
    BinRow bins;
    bins.word = reinterpret_cast<uint32_t*>(base);
    bins.id = reinterpret_cast<uint32_t*>(base + plane);
    bins.p = reinterpret_cast<float*>(base + 2 * plane);
    bins.a = reinterpret_cast<float*>(base + 3 * plane);
    bins.b = reinterpret_cast<float*>(base + 4 * plane);
    uint32_t* kA = reinterpret_cast<uint32_t*>(base + 5 * plane);
    uint32_t* iA = reinterpret_cast<uint32_t*>(base + 6 * plane);
    uint32_t* kB = reinterpret_cast<uint32_t*>(base + 7 * plane);
    uint32_t* iB = reinterpret_cast<uint32_t*>(base + 8 * plane);
    hipLaunchKernelGGL(tlp_rank_sorted_kernel, dim3((unsigned)B), dim3(kRankThreads), 0, st, p, q1, q2, V, s, r,
                       omega1, hdr, bins, kA, iA, kB, iB, row_status);
  } else {
    hipLaunchKernelGGL(tlp_rank_half_kernel, dim3((unsigned)B), dim3(kRankThreads), 0, st, p, q1, q2, V, s, r,
                       omega1, hdr, row_status);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(tlp_lp_kernel, dim3((unsigned)B), dim3(64), 0, st, p, q1, q2, V, s, hdr, omega1, r, w, accept,
                     row_status);
  return hipGetLastError();
}

hipError_t launch_select_tlp(const float* p, const float* q1, const float* q2, const int32_t* drafts, const float* u,
                             uint64_t seed, uint64_t offset, int64_t B, int64_t V, int s, int tail,
                             const int32_t* omega1, const double* w, int32_t* sel_index, int32_t* sel_token,
                             int32_t* row_status, hipStream_t st) {
  if (!q2) q2 = q1;
  const unsigned blocks = (unsigned)((B + 255) / 256);
  hipLaunchKernelGGL(tlp_select_kernel, dim3(blocks), dim3(256), 0, st, p, q1, q2, drafts, u, seed, offset, B, V, s,
                     tail, omega1, w, sel_index, sel_token, row_status);
  return hipGetLastError();
}

}  // namespace mdss
