// Internal declarations of the gfx950 multi-draft selection library.
// Notation: p = target, q = draft, w = p / q (importance weight).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mdss {

// Per-row record written by the preparation kernel.
struct alignas(32) RowHdr {
  int32_t n;      // support size |{x : q(x) > 0}|
  int32_t scale;  // exponent s: scaled weights w' = w * 2^s
  int32_t mode;   // Mode below
  int32_t flags;  // row status bits found by the preparation
  double q0;      // draft mass of support tokens with p = 0 (zero weight)
  double pad;
};

// How a row's pair sum is evaluated.
enum Mode : int32_t {
  kSkip = 0,    // flagged row (r already set to NaN)
  kDirect = 1,  // one reciprocal per (query, pole)
  kRat4 = 4,    // rational form over chunks of 4 poles
  kRat8 = 8,    // rational form over chunks of 8 poles
};

constexpr int kRowBadProb = 1;
constexpr int kRowBadDraft = 2;
constexpr int kRowSupport = 4;
constexpr int kRowForced = 8;
constexpr int kRowLpLimit = 16;
constexpr int kRowRange = 32;
constexpr int kMaxK = 8;  // direct K-draft selection and its induced distribution

// Workspace layout for mdss_induced_dist.
struct Workspace {
  RowHdr* hdr;      // [B]
  int32_t* idx;     // [B][Sp] compacted token ids (ascending), -1 in the padding
  float* wc;        // [B][Sp] compacted scaled weights w'
  float* qc;        // [B][Sp] compacted draft probabilities
  float* stream;    // [B][ld] pole stream: (w', q) pairs, chunk coefficients, or packed bf16 MFMA operands
  int64_t ld;       // floats per row of the pole stream (8 Sp for K = 2, 2 Sp for K = 3)
  double* part;     // [B][P][Sp] partial sums when the pole range is split, else unused
  int64_t Sp;       // padded compacted row length (multiple of 8)
  int32_t P;        // number of pole-range splits
};

size_t workspace_bytes(int64_t B, int64_t V, int K, int s_max, int P);
void carve_workspace(void* base, int64_t B, int64_t V, int K, int s_max, int P, Workspace* ws);
int choose_splits(int64_t B, int64_t V, int K, int s_max);

hipError_t launch_induced(const float* p, const float* q, int64_t B, int64_t V, int K, int s_max, float* r,
                          int32_t* row_status, const Workspace& ws, hipStream_t st);
size_t workspace_bytes_pair(int64_t B, int64_t V);
hipError_t launch_induced_pair(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, float* r,
                               int32_t* row_status, void* workspace, hipStream_t st);
hipError_t launch_select_pair(const float* p, const float* q1, const float* q2, const int32_t* drafts,
                              const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                              int32_t* sel_index, int32_t* sel_token, int32_t* row_status, hipStream_t st);
hipError_t launch_induced_successive(const float* p, const float* q, int64_t B, int64_t V, int K, float* r_stages,
                                     int32_t* row_status, void* workspace, hipStream_t st);
hipError_t launch_select_successive(const float* p, const float* q, const float* r_stages, const int32_t* drafts,
                                    const float* u_sel, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int K,
                                    int32_t* sel_index, int32_t* sel_token, int32_t* row_status, hipStream_t st);
constexpr int kSuccessiveMaxK = 8;
size_t workspace_bytes_optimum(int64_t B, int64_t V);
size_t workspace_bytes_expsum(int64_t B, int64_t V, int L);
// rsum (nullable): also the residual sums of Algorithm 1 with proposal r, kResParts fp64
// partial sums of max(0, p - r) per kResSub-token sub-tile, [B][ceil(V / kResSub)][kResParts]
// (the layout launch_select_accept_sums reads).  With rsum, row_status (nullable) is set
// to the call's flags rather than OR-ed into.
constexpr int kResSub = 1024;
constexpr int kResParts = 4;
hipError_t launch_induced_expsum(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, int K,
                                 float* r, int32_t* row_status, void* workspace, hipStream_t st,
                                 double* rsum = nullptr);
hipError_t launch_induced_successive_expsum(const float* p, const float* q, int64_t B, int64_t V, int K,
                                            float* r_stages, int32_t* row_status, void* workspace, hipStream_t st);
// The K-draft quadrature with its workspace in the library's fixed device scratch
// array (no allocation); B, V must fit in MDSS_NOALLOC_SCRATCH_BYTES.
hipError_t launch_induced_expsum_noalloc(const float* p, const float* q, int64_t B, int64_t V, int K, float* r,
                                         int32_t* row_status, hipStream_t st);
hipError_t launch_select_accept_sums(const float* p, const float* q, const float* q2, const float* r,
                                     const int32_t* drafts, const float* u, uint64_t seed, uint64_t offset,
                                     int64_t B, int64_t V, int K, int32_t* sel_index, int32_t* sel_token,
                                     int32_t* out_token, uint8_t* accepted, double* residual_mass,
                                     int32_t* row_status, void* workspace, hipStream_t st);
// rsum (nullable): the summed form, the residual sums in the layout above; row_status set.
hipError_t launch_induced_topk_expsum(const float* p, const float* q, int64_t B, int64_t V, int K, int s_max,
                                      float* r, int32_t* row_status, hipStream_t st, double* rsum = nullptr);
// The top-s summed form and the draw from its sums (selection and Algorithm 1 as
// launch_select_accept_sums) in one launch.
hipError_t launch_step_topk_expsum(const float* p, const float* q, const int32_t* drafts, const float* u, uint64_t seed,
                                   uint64_t offset, int64_t B, int64_t V, int K, int s_max, float* r,
                                   int32_t* sel_index, int32_t* sel_token, int32_t* out_token, uint8_t* accepted,
                                   double* residual_mass, int32_t* row_status, double* rsum, hipStream_t st);
hipError_t launch_alphabet_truncate(const float* p, int64_t B, int64_t V, int m, float* pt, double* mass0,
                                    int32_t* row_status, hipStream_t st);
hipError_t launch_alphabet_post(const float* p, const float* pt, const double* mass0, const int32_t* token,
                                const float* u2, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                                int32_t* out_token, uint8_t* kept, hipStream_t st);
hipError_t launch_optimum(const float* p, const float* q, int64_t B, int64_t V, int K, double* pstar, int32_t* kstar,
                          int32_t* row_status, void* workspace, hipStream_t st);
hipError_t launch_acceptance(const float* p, const float* r, int64_t B, int64_t V, double* out, int32_t* row_status,
                             hipStream_t st);
size_t workspace_bytes_tlp(int64_t B, int64_t V, int tail);
hipError_t launch_tlp(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, int s, int tail,
                      float* r, int32_t* omega1, double* w, double* accept, int32_t* row_status, void* workspace,
                      hipStream_t st);
hipError_t launch_select_tlp(const float* p, const float* q1, const float* q2, const int32_t* drafts, const float* u,
                             uint64_t seed, uint64_t offset, int64_t B, int64_t V, int s, int tail,
                             const int32_t* omega1, const double* w, int32_t* sel_index, int32_t* sel_token,
                             int32_t* row_status, hipStream_t st);
hipError_t launch_select(const float* p, const float* q, const int32_t* drafts, const float* u, uint64_t seed,
                         uint64_t offset, int64_t B, int64_t V, int K, int32_t* sel_index, int32_t* sel_token,
                         int32_t* row_status, hipStream_t st);
size_t workspace_bytes_accept(int64_t B, int64_t V);
hipError_t launch_accept(const float* p, const float* r, const int32_t* sel_token, const float* u, uint64_t seed,
                         uint64_t offset, int64_t B, int64_t V, int32_t* out_token, uint8_t* accepted,
                         float* residual, double* residual_mass, int32_t* row_status, void* workspace,
                         hipStream_t st);
hipError_t launch_select_accept(const float* p, const float* q, const float* q2, const float* r,
                                const int32_t* drafts, const float* u, uint64_t seed, uint64_t offset, int64_t B,
                                int64_t V, int K, int32_t* sel_index, int32_t* sel_token, int32_t* out_token,
                                uint8_t* accepted, float* residual, double* residual_mass, int32_t* row_status,
                                void* workspace, hipStream_t st);

// ---------------------------------------------------------------- device helpers
__device__ __forceinline__ bool bad_prob(float v) { return !(v >= 0.0f) || isinf(v); }

// The residual of Algorithm 1 at one token, max(0, p - r), in fp64 (exact for fp32 p and r).
__device__ __forceinline__ double residual_of(float pv, float rv) {
  const double d = (double)pv - (double)rv;
  return d > 0.0 ? d : 0.0;
}

// fp64 lane moves by DPP (each 32-bit half moved the same way)
template <int CTRL, int ROW_MASK = 0xF, bool BOUND_ZERO = false>
__device__ __forceinline__ double dpp64(double x) {
  const uint64_t v = __double_as_longlong(x);
  const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)v, CTRL, ROW_MASK, 0xF, BOUND_ZERO);
  const uint32_t hi = __builtin_amdgcn_update_dpp(0u, (uint32_t)(v >> 32), CTRL, ROW_MASK, 0xF, BOUND_ZERO);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// x + the value of the partner lane of a gfx950 row swap (ROW) or half swap
template <bool ROW>
__device__ __forceinline__ double swap_sum64(double x) {
  const uint64_t v = __double_as_longlong(x);
  const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  const auto a = ROW ? __builtin_amdgcn_permlane16_swap(lo, lo, false, false)
                     : __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
  const auto c = ROW ? __builtin_amdgcn_permlane16_swap(hi, hi, false, false)
                     : __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  return __longlong_as_double((long long)(((uint64_t)c[0] << 32) | a[0])) +
         __longlong_as_double((long long)(((uint64_t)c[1] << 32) | a[1]));
}
// Sum over the 64 lanes of a wave, in every lane: quad permutations and row
// rotations within each 16-lane row, then the row and half swaps (all lanes active).
__device__ __forceinline__ double wave_sum_dpp(double x) {
  x += dpp64<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp64<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp64<0x124>(x);  // row_ror:4
  x += dpp64<0x128>(x);  // row_ror:8
  x = swap_sum64<true>(x);
  return swap_sum64<false>(x);
}
// Inclusive prefix sum over the 64 lanes of a wave (fixed order): Hillis-Steele
// within each 16-lane row by DPP row shifts (lanes shifted in from outside the
// row read 0), then each row adds the totals of the rows before it, read from
// lanes 15, 31 and 47.
__device__ __forceinline__ double wave_inclusive_scan_dpp(double x, int lane) {
  x += dpp64<0x111, 0xF, true>(x);  // row_shr:1
  x += dpp64<0x112, 0xF, true>(x);  // row_shr:2
  x += dpp64<0x114, 0xF, true>(x);  // row_shr:4
  x += dpp64<0x118, 0xF, true>(x);  // row_shr:8
  const uint64_t v = __double_as_longlong(x);
  const auto rd = [&](int l) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, l), hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), l);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
  };
  const double t0 = rd(15), t1 = rd(31), t2 = rd(47);
  const int row = lane >> 4;
  const double c01 = t0 + t1;
  const double carry = row == 0 ? 0.0 : (row == 1 ? t0 : (row == 2 ? c01 : c01 + t2));
  return row == 0 ? x : x + carry;
}


// Philox4x32-10 (Salmon et al., SC'11): ten rounds of the 4x32 S-box with the
// published multipliers and Weyl key increments.
__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t lo0 = 0xD2511F53u * c[0], hi0 = __umulhi(0xD2511F53u, c[0]);
    const uint32_t lo1 = 0xCD9E8D57u * c[2], hi1 = __umulhi(0xCD9E8D57u, c[2]);
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

// Uniform j (0: select, 1: accept, 2: residual) of a position: from the
// caller's array, else from Philox(seed, offset + b).
__device__ __forceinline__ void position_uniforms(const float* u, uint64_t seed, uint64_t offset, int64_t b,
                                                  float out[3]) {
  if (u) {
    out[0] = u[b * 3 + 0];
    out[1] = u[b * 3 + 1];
    out[2] = u[b * 3 + 2];
    return;
  }
  const uint64_t pos = offset + (uint64_t)b;
  uint32_t c[4] = {(uint32_t)pos, (uint32_t)(pos >> 32), 0u, 0u};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
  for (int j = 0; j < 3; ++j) out[j] = (float)(c[j] >> 8) * 5.9604644775390625e-8f;  // 2^-24
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ int wave_sum_int(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fminf(v, __shfl_xor(v, off, 64));
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}
// Inclusive prefix sum across the 64 lanes of a wave (Hillis-Steele, fixed order).
__device__ __forceinline__ double wave_inclusive_scan(double v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}
__device__ __forceinline__ int wave_inclusive_scan_int(int v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

}  // namespace mdss
