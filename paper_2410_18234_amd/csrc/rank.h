// Per-row ranking and reverse scan on gfx950, shared by the truncated linear
// program and the optimal-acceptance diagnostics.
//
// One workgroup of 1024 threads per row.  Each token gets a 32-bit word whose
// ascending order is the ranking (ties: ascending token id).  Pass 1 reads the
// row, checks it, sums two row totals and counts the top 8 bits of the words
// per wave (stable); pass 2 scatters (word, id, three values) into 256 bins;
// pass 3 takes the bins from the last-ranked down, groups consecutive bins of at
// most kGroup entries, sorts each group in LDS with stable 8-bit LSD passes (a
// single bin above kGroup entries: stable passes in global memory on its lower
// 24 bits), gathers the group's values into LDS and scans it in reverse rank
// order, giving every entry the two masses ranked after it.  What is done with
// each entry is the Spec's.
#pragma once

#include "common.h"

#include <math.h>

namespace mdss {
namespace {

constexpr int kRankThreads = 1024;
constexpr int kRankWaves = kRankThreads / 64;
constexpr int kGroup = 8192;  // entries sorted in LDS at once
constexpr int kStride = kGroup / kRankThreads;

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

// Bin-ordered copy of a row made by pass 2 (structure of arrays).
struct BinRow {
  uint32_t* word;
  uint32_t* id;
  float* v0;
  float* v1;
  float* v2;
};

// Workspace planes of the ranking: 5 for the bin-ordered copy, 4 for a bin
// above the LDS capacity; each [B][V] 32-bit words.
constexpr int kRankPlanes = 9;

struct RankPlanes {
  BinRow bins;
  uint32_t *kA, *iA, *kB, *iB;
};

// Reverse scan of a ranked chunk whose entries are staged in LDS in rank order
// (V0, V1, V2, ID; g < G <= kGroup, rank first_rank + g): each thread owns E
// consecutive ranks, the block scan gives every entry the two masses
// (Spec::masses) ranked after it, and Spec::visit sees each entry with them.
template <class Spec>
__device__ __forceinline__ void scan_staged(int G, uint32_t first_rank, const typename Spec::Row& row,
                                            typename Spec::State& state, double* c1, double* c2, double* sa,
                                            double* sb, const float* V0, const float* V1, const float* V2,
                                            const uint32_t* ID) {
  const int E = (G + kRankThreads - 1) / kRankThreads;
  const int g0 = min(G, (int)threadIdx.x * E), g1 = min(G, g0 + E);
  double l1 = 0.0, l2 = 0.0;  // this thread's masses (consecutive ranks)
  for (int g = g0; g < g1; ++g) {
    double m1, m2;
    Spec::masses(row, first_rank + (uint32_t)g, V0[g], V1[g], V2[g], &m1, &m2);
    l1 += m1;
    l2 += m2;
  }
  double e1, e2, t1, t2;
  block_exclusive_suffix2(l1, l2, &e1, &e2, &t1, &t2, sa, sb);
  double s1 = *c1 + e1, s2 = *c2 + e2;  // masses ranked after the entry being visited
  for (int g = g1 - 1; g >= g0; --g) {
    const uint32_t rank = first_rank + (uint32_t)g;
    Spec::visit(row, state, rank, (int)ID[g], V0[g], V1[g], V2[g], s1, s2);
    double m1, m2;
    Spec::masses(row, rank, V0[g], V1[g], V2[g], &m1, &m2);
    s1 += m1;
    s2 += m2;
  }
  *c1 += t1;
  *c2 += t2;
  __syncthreads();  // the staging arrays are reused by the next chunk
}

// A group sorted in LDS: inv[i] = rank within the group of bin-order entry i
// (i < G).  The entries are read in bin order (coalesced) and written to their
// rank's slot of the staging arrays (`inv` may alias one of them), then scanned.
template <class Spec>
__device__ __forceinline__ void scan_group(const uint32_t* inv, int G, uint32_t g_lo, const BinRow& br,
                                           const typename Spec::Row& row, typename Spec::State& state, double* c1,
                                           double* c2, double* sa, double* sb, float* V0, float* V1, float* V2,
                                           uint32_t* ID) {
  uint32_t slot[kStride];
#pragma unroll
  for (int k = 0; k < kStride; ++k) {
    const int i = (int)threadIdx.x + k * kRankThreads;
    slot[k] = i < G ? inv[i] : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kStride; ++k) {
    const int i = (int)threadIdx.x + k * kRankThreads;
    if (i < G) {
      const uint32_t at = g_lo + (uint32_t)i;
      V0[slot[k]] = br.v0[at];
      V1[slot[k]] = br.v1[at];
      V2[slot[k]] = br.v2[at];
      ID[slot[k]] = br.id[at];
    }
  }
  __syncthreads();
  scan_staged<Spec>(G, g_lo, row, state, c1, c2, sa, sb, V0, V1, V2, ID);
}

// A chunk of a bin sorted in global memory: sorted[g] = bin-order index of
// rank first_rank + g; the entries are gathered (thread-strided, many loads in
// flight) into the staging arrays, then scanned.
template <class Spec>
__device__ __forceinline__ void scan_chunk(const uint32_t* sorted, int G, uint32_t first_rank, uint32_t bin_base,
                                           const BinRow& br, const typename Spec::Row& row,
                                           typename Spec::State& state, double* c1, double* c2, double* sa,
                                           double* sb, float* V0, float* V1, float* V2, uint32_t* ID) {
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
      V0[g] = br.v0[at[k]];
      V1[g] = br.v1[at[k]];
      V2[g] = br.v2[at[k]];
      ID[g] = br.id[at[k]];
    }
  }
  __syncthreads();
  scan_staged<Spec>(G, first_rank, row, state, c1, c2, sa, sb, V0, V1, V2, ID);
}

// The ranking kernel.  Spec provides:
//   Args, Row, State; Row row(const Args&, int64_t b, int64_t V);
//   const float* in0/in1/in2 in Row (the three values read per token);
//   uint32_t word(float v0, float v1, float v2);
//   void set_totals(Row&, double sum_v0, double sum_v1);
//   void masses(const Row&, uint32_t rank, float v0, float v1, float v2, double* m1, double* m2);
//   void visit(const Row&, State&, uint32_t rank, int id, float v0, float v1, float v2, double s1, double s2);
//   void flag(const Row&, int64_t V, int flags);  (all threads; the row failed its check)
//   void finish(const Row&, State&, double c1, double c2, double* red);  (all threads)
template <class Spec>
__global__ __launch_bounds__(kRankThreads) void rank_scan_kernel(typename Spec::Args args, int64_t V,
                                                                 RankPlanes planes) {
  __shared__ uint32_t cnt[kRankWaves][256];
  __shared__ uint32_t tot[256], bin_cnt[256], bin_start[256];
  __shared__ uint32_t kx[2][kGroup], ix[2][kGroup];
  __shared__ double sa[kRankWaves], sb[kRankWaves];
  __shared__ int red[kRankWaves];
  __shared__ int flag;
  const int64_t b = blockIdx.x;
  typename Spec::Row row = Spec::row(args, b, V);
  const float* x0 = row.in0;
  const float* x1 = row.in1;
  const float* x2 = row.in2;
  const int n = (int)V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const BinRow br = {planes.bins.word + b * V, planes.bins.id + b * V, planes.bins.v0 + b * V,
                     planes.bins.v1 + b * V, planes.bins.v2 + b * V};
  int lo, hi;
  wave_segment(n, &lo, &hi);
  constexpr int kBatch = 4;
  // pass 1: validity, totals and per-wave counts of the top digit
  for (int d = lane; d < 256; d += 64) cnt[wave][d] = 0u;
  int bad = 0;
  double t0 = 0.0, t1 = 0.0;
  for (int base = lo; base < hi; base += 64 * kBatch) {
    float r0[kBatch], r1[kBatch], r2[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      r0[j] = i < hi ? x0[i] : 0.0f;
      r1[j] = i < hi ? x1[i] : 0.0f;
      r2[j] = i < hi ? x2[i] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      const uint64_t act = __ballot(i < hi);
      if (!act) break;
      bad |= (bad_prob(r0[j]) || bad_prob(r1[j]) || bad_prob(r2[j])) ? 1 : 0;
      t0 += (double)r0[j];
      t1 += (double)r1[j];
      const uint32_t d = Spec::word(r0[j], r1[j], r2[j]) >> 24;
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
    Spec::flag(row, V, kRowBadProb);
    return;
  }
  Spec::set_totals(row, block_sum(t0, sa), block_sum(t1, sa));
  digit_offsets(cnt, tot, 0u, n, bin_cnt, bin_start, &flag);
  // pass 2: stable scatter into bin order, with the values the scan needs
  for (int base = lo; base < hi; base += 64 * kBatch) {
    float r0[kBatch], r1[kBatch], r2[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      r0[j] = i < hi ? x0[i] : 0.0f;
      r1[j] = i < hi ? x1[i] : 0.0f;
      r2[j] = i < hi ? x2[i] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * 64 + lane;
      const uint64_t act = __ballot(i < hi);
      if (!act) break;
      const uint32_t wd = Spec::word(r0[j], r1[j], r2[j]);
      const uint32_t d = wd >> 24;
      const uint64_t m = match_digit(d, act);
      if (i < hi) {
        const uint32_t pos = cnt[wave][d] + (uint32_t)__popcll(m & lanes_below(lane));
        br.word[pos] = wd;
        br.id[pos] = (uint32_t)i;
        br.v0[pos] = r0[j];
        br.v1[pos] = r1[j];
        br.v2[pos] = r2[j];
        if (lane == __ffsll((long long)m) - 1) cnt[wave][d] += (uint32_t)__popcll(m);
      }
    }
  }
  __syncthreads();
  // pass 3: groups of bins, last-ranked first
  typename Spec::State state;
  double c1 = 0.0, c2 = 0.0;
  float* V0 = reinterpret_cast<float*>(kx[0]);
  float* V1 = reinterpret_cast<float*>(kx[1]);
  float* V2 = reinterpret_cast<float*>(ix[0]);
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
      // inverse permutation (rank of each bin-order entry) into the free index buffer
      for (uint32_t g = threadIdx.x; g < G; g += kRankThreads) ix[cur ^ 1][ix[cur][g]] = g;
      __syncthreads();
      scan_group<Spec>(ix[cur ^ 1], (int)G, g_lo, br, row, state, &c1, &c2, sa, sb, V0, V1, V2, ix[1]);
    } else {
      // one bin above the LDS capacity: its words share the top digit
      uint32_t* ka = planes.kA + b * V;
      uint32_t* ia = planes.iA + b * V;
      uint32_t* kb = planes.kB + b * V;
      uint32_t* ib = planes.iB + b * V;
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
      const int chunks = (int)((G + kGroup - 1) / kGroup);
      for (int c = chunks - 1; c >= 0; --c) {
        const uint32_t c0 = (uint32_t)c * kGroup;
        const int Gc = (int)min((uint32_t)kGroup, G - c0);
        scan_chunk<Spec>(i_in + c0, Gc, g_lo + c0, g_lo, br, row, state, &c1, &c2, sa, sb, V0, V1, V2, ix[1]);
      }
    }
    dh = dl - 1;
  }
  Spec::finish(row, state, c1, c2, sa);
}

inline size_t rank_align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline size_t rank_workspace_bytes(int64_t B, int64_t V) {
  return kRankPlanes * rank_align256((size_t)B * (size_t)V * sizeof(uint32_t));
}

inline RankPlanes carve_rank_planes(void* base_ptr, int64_t B, int64_t V) {
  char* base = static_cast<char*>(base_ptr);
  const size_t plane = rank_align256((size_t)B * (size_t)V * sizeof(uint32_t));
  RankPlanes r;
  r.bins.word = reinterpret_cast<uint32_t*>(base);
  r.bins.id = reinterpret_cast<uint32_t*>(base + plane);
  r.bins.v0 = reinterpret_cast<float*>(base + 2 * plane);
  r.bins.v1 = reinterpret_cast<float*>(base + 3 * plane);
  r.bins.v2 = reinterpret_cast<float*>(base + 4 * plane);
  r.kA = reinterpret_cast<uint32_t*>(base + 5 * plane);
  r.iA = reinterpret_cast<uint32_t*>(base + 6 * plane);
  r.kB = reinterpret_cast<uint32_t*>(base + 7 * plane);
  r.iB = reinterpret_cast<uint32_t*>(base + 8 * plane);
  return r;
}

}  // namespace
}  // namespace mdss
