// Optimal acceptance diagnostics, gfx950.
//
// Theorem 3 (K = 2 drafts from q): P* = min over token sets S of
// P(S) + Q(S^c)^2 + 2 Q(S) Q(S^c) = Qt^2 + min_S (P(S) - Q(S)^2), with P, Q
// the target / draft masses and Qt the draft mass of the row; Remark 2's
// K-draft form (conjectured for K > 2) replaces the power 2 by K.  By strict
// convexity of x^K a minimising S is {w < threshold} for w = p / q, so the
// minimum over all 2^V sets equals the minimum over the V + 1 prefixes of the
// tokens ordered by w ascending (q = 0 last).  The rank scan orders each row by
// w (fp64 ratio rounded once to fp32; ties by lower id) and evaluates every
// prefix from the masses ranked after each entry: P_k = Pt - (p mass after),
// Q_k = Qt - (q mass after).
//
// Notation: p = target, q = draft.
#include "rank.h"

namespace mdss {

namespace {

__device__ __forceinline__ double ipow(double x, int K) {
  double y = 1.0;
  for (int i = 0; i < K; ++i) y *= x;
  return y;
}

struct OptSpec {
  struct Args {
    const float *p, *q;
    double* pstar;
    int32_t* kstar;
    int32_t* row_status;
    int K;
  };
  struct Row {
    const float *in0, *in1, *in2;
    double* pstar;
    int32_t* kstar;
    int32_t* row_status;
    int64_t b;
    double Pt, Qt;
    int K;
  };
  struct State {
    double best = __longlong_as_double(0x7ff0000000000000ll);  // +inf
    uint32_t k = 0xffffffffu;                                   // prefix length attaining it
  };
  static __device__ __forceinline__ Row row(const Args& a, int64_t b, int64_t V) {
    Row r;
    r.in0 = a.p + b * V;
    r.in1 = a.q + b * V;
    r.in2 = r.in1;
    r.pstar = a.pstar;
    r.kstar = a.kstar;
    r.row_status = a.row_status;
    r.b = b;
    r.Pt = r.Qt = 0.0;
    r.K = a.K;
    return r;
  }
  // w = p / q ascending; q = 0 (and a ratio above the fp32 range) rank last
  static __device__ __forceinline__ uint32_t word(float p, float q, float) {
    const float w = q > 0.0f ? (float)((double)p / (double)q) : __int_as_float(0x7f800000);
    return __float_as_uint(w + 0.0f);
  }
  static __device__ __forceinline__ void set_totals(Row& r, double pt, double qt) {
    r.Pt = pt;
    r.Qt = qt;
  }
  static __device__ __forceinline__ void masses(const Row&, uint32_t, float p, float q, float, double* m1,
                                                double* m2) {
    *m1 = (double)p;
    *m2 = (double)q;
  }
  static __device__ __forceinline__ void visit(const Row& r, State& st, uint32_t rank, int, float, float, float,
                                               double s1, double s2) {
    const double f = (r.Pt - s1) + ipow(r.Qt, r.K) - ipow(r.Qt - s2, r.K);
    const uint32_t k = rank + 1u;
    if (f < st.best || (f == st.best && k < st.k)) {
      st.best = f;
      st.k = k;
    }
  }
  static __device__ __forceinline__ void flag(const Row& r, int64_t, int flags) {
    if (threadIdx.x == 0) {
      r.pstar[r.b] = __longlong_as_double(0x7ff8000000000000ll);
      if (r.kstar) r.kstar[r.b] = -1;
      if (r.row_status) r.row_status[r.b] |= flags;
    }
  }
  static __device__ __forceinline__ void finish(const Row& r, State& st, double, double, double* red) {
    // block minimum of (value, prefix length), smaller length on equal values
    double v = st.best;
    uint32_t k = st.k;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const double ov = __shfl_xor(v, off, 64);
      const uint32_t ok = __shfl_xor(k, off, 64);
      if (ov < v || (ov == v && ok < k)) {
        v = ov;
        k = ok;
      }
    }
    __shared__ uint32_t redk[kRankWaves];
    if ((threadIdx.x & 63) == 0) {
      red[threadIdx.x >> 6] = v;
      redk[threadIdx.x >> 6] = k;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      double bv = ipow(r.Qt, r.K);  // the empty prefix
      uint32_t bk = 0;
      for (int w = 0; w < kRankWaves; ++w)
        if (red[w] < bv || (red[w] == bv && redk[w] < bk)) {
          bv = red[w];
          bk = redk[w];
        }
      r.pstar[r.b] = bv;
      if (r.kstar) r.kstar[r.b] = (int32_t)bk;
    }
  }
};

// sum over the row of min(p, r), fp64, in a fixed order; NaN if the row is bad
constexpr int kAccThreads = 1024;
__global__ __launch_bounds__(kAccThreads) void acceptance_kernel(const float* __restrict__ p,
                                                                 const float* __restrict__ r, int64_t V,
                                                                 double* __restrict__ out,
                                                                 int32_t* __restrict__ row_status) {
  __shared__ double red[kAccThreads / 64];
  __shared__ int bad_w[kAccThreads / 64];
  const int64_t b = blockIdx.x;
  const float* pb = p + b * V;
  const float* rb = r + b * V;
  double acc = 0.0;
  int bad = 0;
  constexpr int kU = 4;
  for (int64_t i0 = threadIdx.x; i0 < V; i0 += kU * kAccThreads) {
    float pv[kU], rv[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int64_t i = i0 + (int64_t)u * kAccThreads;
      pv[u] = i < V ? pb[i] : 0.0f;
      rv[u] = i < V ? rb[i] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      bad |= (bad_prob(pv[u]) || bad_prob(rv[u])) ? 1 : 0;
      acc += fmin((double)pv[u], (double)rv[u]);
    }
  }
  acc = wave_sum(acc);
  bad = __ballot(bad) != 0ull;
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = acc;
    bad_w[threadIdx.x >> 6] = bad;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int any = 0;
    double t = 0.0;
    for (int w = 0; w < kAccThreads / 64; ++w) {
      any |= bad_w[w];
      t += red[w];
    }
    out[b] = any ? __longlong_as_double(0x7ff8000000000000ll) : t;
    if (any && row_status) row_status[b] |= kRowBadProb;
  }
}

}  // namespace

size_t workspace_bytes_optimum(int64_t B, int64_t V) { return rank_workspace_bytes(B, V); }

hipError_t launch_optimum(const float* p, const float* q, int64_t B, int64_t V, int K, double* pstar, int32_t* kstar,
                          int32_t* row_status, void* workspace, hipStream_t st) {
  OptSpec::Args args = {p, q, pstar, kstar, row_status, K};
  hipLaunchKernelGGL(rank_scan_kernel<OptSpec>, dim3((unsigned)B), dim3(kRankThreads), 0, st, args, V,
                     carve_rank_planes(workspace, B, V));
  return hipGetLastError();
}

hipError_t launch_acceptance(const float* p, const float* r, int64_t B, int64_t V, double* out, int32_t* row_status,
                             hipStream_t st) {
  hipLaunchKernelGGL(acceptance_kernel, dim3((unsigned)B), dim3(kAccThreads), 0, st, p, r, V, out, row_status);
  return hipGetLastError();
}

}  // namespace mdss
