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
#include "rank.h"

#include <math.h>

namespace mdss {

namespace {

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

// ---------------------------------------------------------------- SORTED tail
// The ranking of Algorithm 2 on the rank scan: values (p, q1, q2); the scan
// masses are (q1, q2) of the Omega_2 entries; an Omega_1 entry (rank < s) is
// recorded in omega1, every Omega_2 entry k gets r(k) = q1 q2 + q2 S1 + q1 S2.
struct TlpSpec {
  struct Args {
    const float *p, *q1, *q2;
    float* r;
    int32_t* omega1;
    TlpHdr* hdr;
    int32_t* row_status;
    int s;
  };
  struct Row {
    const float *in0, *in1, *in2;
    float* rb;
    int32_t* omega1;
    TlpHdr* hdr;
    int32_t* row_status;
    int64_t b, V;
    int s;
  };
  struct State {
    double acc = 0.0;  // sum over Omega_2 of min(p, r)
  };
  static __device__ __forceinline__ Row row(const Args& a, int64_t b, int64_t V);
  static __device__ __forceinline__ uint32_t word(float p, float q1, float q2) { return rank_word(p, q1, q2); }
  static __device__ __forceinline__ void set_totals(Row&, double, double) {}
  static __device__ __forceinline__ void masses(const Row& r, uint32_t rank, float, float q1, float q2, double* m1,
                                                double* m2) {
    const bool om1 = rank < (uint32_t)r.s;
    *m1 = om1 ? 0.0 : (double)q1;
    *m2 = om1 ? 0.0 : (double)q2;
  }
  static __device__ __forceinline__ void visit(const Row& r, State& st, uint32_t rank, int id, float p, float q1,
                                               float q2, double s1, double s2) {
    if (rank < (uint32_t)r.s) {
      r.omega1[r.b * r.s + rank] = id;
      return;
    }
    const double av = (double)q1, bv = (double)q2;
    const double rv = av * bv + bv * s1 + av * s2;
    r.rb[id] = (float)rv;
    st.acc += fmin((double)p, rv);
  }
  static __device__ __forceinline__ void flag(const Row& r, int64_t V, int flags) {
    flag_row(r.b, V, r.s, r.rb, r.omega1, r.hdr, r.row_status, flags);
  }
  static __device__ __forceinline__ void finish(const Row& r, State& st, double c1, double c2, double* red) {
    const int se = (int)min((int64_t)r.s, r.V);
    if ((int)threadIdx.x >= se && (int)threadIdx.x < r.s) r.omega1[r.b * r.s + threadIdx.x] = -1;
    const double acc = block_sum(st.acc, red);
    if (threadIdx.x == 0) {
      TlpHdr h = {};
      h.s_eff = se;
      h.a_tail = c1;
      h.b_tail = c2;
      h.tail_accept = acc;
      r.hdr[r.b] = h;
    }
  }
};

__device__ __forceinline__ TlpSpec::Row TlpSpec::row(const Args& a, int64_t b, int64_t V) {
  Row r;
  r.in0 = a.p + b * V;
  r.in1 = a.q1 + b * V;
  r.in2 = a.q2 + b * V;
  r.rb = a.r + b * V;
  r.omega1 = a.omega1;
  r.hdr = a.hdr;
  r.row_status = a.row_status;
  r.b = b;
  r.V = V;
  r.s = a.s;
  return r;
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

size_t workspace_bytes_tlp(int64_t B, int64_t V, int tail) {
  size_t bytes = align256((size_t)B * sizeof(TlpHdr));
  if (tail == kTailSorted) bytes += rank_workspace_bytes(B, V);
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
    TlpSpec::Args args = {p, q1, q2, r, omega1, hdr, row_status, s};
    hipLaunchKernelGGL(rank_scan_kernel<TlpSpec>, dim3((unsigned)B), dim3(kRankThreads), 0, st, args, V,
                       carve_rank_planes(base, B, V));
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
