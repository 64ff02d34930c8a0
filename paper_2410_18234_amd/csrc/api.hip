// C ABI entry points: argument validation and launches on the caller's stream.
#include "mdss.h"

#include <hip/hip_runtime.h>

#include "common.h"

namespace {

constexpr int32_t kAbiVersion = 1;

// B = 0 is an empty batch: after the shape and parameter checks an entry point
// returns MDSS_OK without reading, writing or launching anything.
mdss_status check_shape(int64_t B, int64_t V) {
  if (B < 0 || B > MDSS_MAX_B || V < 2 || V > MDSS_MAX_V) return MDSS_ESHAPE;
  return MDSS_OK;
}

bool workspace_ok(const void* ws, size_t bytes, size_t need) {
  return ws && bytes >= need && (reinterpret_cast<uintptr_t>(ws) % 256) == 0;
}

mdss_status check_k(int32_t K, int32_t s_max) {
  if (K != 2 && K != 3) return MDSS_EUNSUPPORTED;
  if (K == 3 && (s_max < 1 || s_max > MDSS_K3_MAX_SUPPORT)) return MDSS_EUNSUPPORTED;
  return MDSS_OK;
}

mdss_status from_hip(hipError_t e) { return e == hipSuccess ? MDSS_OK : MDSS_EDEVICE; }

}  // namespace

extern "C" {

int32_t mdss_abi_version(void) { return kAbiVersion; }

const char* mdss_status_string(mdss_status s) {
  switch (s) {
    case MDSS_OK: return "ok";
    case MDSS_EINVAL: return "invalid argument (null pointer or bad value)";
    case MDSS_ESHAPE: return "invalid shape (B outside [0, MDSS_MAX_B] or V outside [2, MDSS_MAX_V])";
    case MDSS_EUNSUPPORTED: return "unsupported configuration (K out of range, K = 3 with s_max out of range, or s outside [1, MDSS_TLP_MAX_S])";
    case MDSS_EDEVICE: return "HIP error while launching";
    case MDSS_EWORKSPACE: return "workspace missing or too small (allocation-free call: sizes beyond MDSS_NOALLOC_SCRATCH_BYTES)";
  }
  return "unknown status";
}

size_t mdss_workspace_bytes(int64_t B, int64_t V, int32_t K, int32_t s_max) {
  if (check_shape(B, V) != MDSS_OK || check_k(K, s_max) != MDSS_OK || B == 0) return 0;
  const int P = mdss::choose_splits(B, V, K, s_max);
  return mdss::workspace_bytes(B, V, K, s_max, P);
}

mdss_status mdss_induced_dist(const float* p, const float* q, int64_t B, int64_t V, int32_t K, int32_t s_max,
                              float* r, int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream) {
  mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if ((s = check_k(K, s_max)) != MDSS_OK) return s;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r) return MDSS_EINVAL;
  const int P = mdss::choose_splits(B, V, K, s_max);
  const size_t need = mdss::workspace_bytes(B, V, K, s_max, P);
  if (!workspace_ok(workspace, workspace_bytes, need)) return MDSS_EWORKSPACE;
  mdss::Workspace ws;
  mdss::carve_workspace(workspace, B, V, K, s_max, P, &ws);
  return from_hip(mdss::launch_induced(p, q, B, V, K, s_max, r, row_status, ws, static_cast<hipStream_t>(stream)));
}

size_t mdss_workspace_bytes_pair(int64_t B, int64_t V) {
  if (check_shape(B, V) != MDSS_OK || B == 0) return 0;
  return mdss::workspace_bytes_pair(B, V);
}

mdss_status mdss_induced_dist_pair(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, float* r,
                                   int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (B == 0) return MDSS_OK;
  if (!p || !q1 || !q2 || !r) return MDSS_EINVAL;
  const size_t need = mdss::workspace_bytes_pair(B, V);
  if (!workspace_ok(workspace, workspace_bytes, need)) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_pair(p, q1, q2, B, V, r, row_status, workspace,
                                            static_cast<hipStream_t>(stream)));
}

mdss_status mdss_select_intermediate_pair(const float* p, const float* q1, const float* q2, const int32_t* drafts,
                                          const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                                          int32_t* sel_index, int32_t* sel_token, int32_t* row_status,
                                          void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (B == 0) return MDSS_OK;
  if (!p || !q1 || !q2 || !drafts || !sel_index || !sel_token) return MDSS_EINVAL;
  return from_hip(mdss::launch_select_pair(p, q1, q2, drafts, u, seed, offset, B, V, sel_index, sel_token,
                                           row_status, static_cast<hipStream_t>(stream)));
}

size_t mdss_workspace_bytes_successive(int64_t B, int64_t V) {
  if (check_shape(B, V) != MDSS_OK || B == 0) return 0;
  return mdss::workspace_bytes_pair(B, V);
}

mdss_status mdss_induced_dist_successive(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                         float* r_stages, int32_t* row_status, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (K < 2 || K > MDSS_SUCCESSIVE_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r_stages) return MDSS_EINVAL;
  const size_t need = mdss::workspace_bytes_pair(B, V);
  if (!workspace_ok(workspace, workspace_bytes, need)) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_successive(p, q, B, V, K, r_stages, row_status, workspace,
                                                  static_cast<hipStream_t>(stream)));
}

mdss_status mdss_select_successive(const float* p, const float* q, const float* r_stages, const int32_t* drafts,
                                   const float* u_sel, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                                   int32_t K, int32_t* sel_index, int32_t* sel_token, int32_t* row_status,
                                   void* stream) {
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (K < 2 || K > MDSS_SUCCESSIVE_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !drafts || !sel_index || !sel_token) return MDSS_EINVAL;
  if (K > 2 && !r_stages) return MDSS_EINVAL;
  return from_hip(mdss::launch_select_successive(p, q, r_stages, drafts, u_sel, seed, offset, B, V, K, sel_index,
                                                 sel_token, row_status, static_cast<hipStream_t>(stream)));
}

mdss_status mdss_truncate_alphabet(const float* p, int64_t B, int64_t V, int32_t m, float* p_trunc, double* mass0,
                                   int32_t* row_status, void* stream) {
  if (m < 1) return MDSS_EINVAL;
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (B == 0) return MDSS_OK;
  if (!p || !p_trunc || !mass0) return MDSS_EINVAL;
  return from_hip(mdss::launch_alphabet_truncate(p, B, V, m, p_trunc, mass0, row_status,
                                                 static_cast<hipStream_t>(stream)));
}

mdss_status mdss_alphabet_post(const float* p, const float* p_trunc, const double* mass0, const int32_t* token,
                               const float* u2, uint64_t seed, uint64_t offset, int64_t B, int64_t V,
                               int32_t* out_token, uint8_t* kept, void* stream) {
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (B == 0) return MDSS_OK;
  if (!p || !p_trunc || !mass0 || !token || !out_token || !kept) return MDSS_EINVAL;
  return from_hip(mdss::launch_alphabet_post(p, p_trunc, mass0, token, u2, seed, offset, B, V, out_token, kept,
                                             static_cast<hipStream_t>(stream)));
}

size_t mdss_workspace_bytes_optimum(int64_t B, int64_t V) {
  if (check_shape(B, V) != MDSS_OK || B == 0) return 0;
  return mdss::workspace_bytes_optimum(B, V);
}

mdss_status mdss_optimal_acceptance(const float* p, const float* q, int64_t B, int64_t V, int32_t K, double* pstar,
                                    int32_t* kstar, int32_t* row_status, void* workspace, size_t workspace_bytes,
                                    void* stream) {
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (K < 2 || K > MDSS_OPTIMUM_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !pstar) return MDSS_EINVAL;
  const size_t need = mdss::workspace_bytes_optimum(B, V);
  if (!workspace_ok(workspace, workspace_bytes, need)) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_optimum(p, q, B, V, K, pstar, kstar, row_status, workspace,
                                       static_cast<hipStream_t>(stream)));
}

mdss_status mdss_acceptance(const float* p, const float* r, int64_t B, int64_t V, double* accept,
                            int32_t* row_status, void* stream) {
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (B == 0) return MDSS_OK;
  if (!p || !r || !accept) return MDSS_EINVAL;
  return from_hip(mdss::launch_acceptance(p, r, B, V, accept, row_status, static_cast<hipStream_t>(stream)));
}

size_t mdss_workspace_bytes_tlp(int64_t B, int64_t V, int32_t tail) {
  if (check_shape(B, V) != MDSS_OK || (tail != MDSS_TLP_SORTED && tail != MDSS_TLP_HALF) || B == 0) return 0;
  return mdss::workspace_bytes_tlp(B, V, tail);
}

mdss_status mdss_truncated_lp(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, int32_t s,
                              int32_t tail, float* r, int32_t* omega1, double* w, double* accept,
                              int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream) {
  if (tail != MDSS_TLP_SORTED && tail != MDSS_TLP_HALF) return MDSS_EINVAL;
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (s < 1 || s > MDSS_TLP_MAX_S) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q1 || !r || !omega1 || !w) return MDSS_EINVAL;
  const size_t need = mdss::workspace_bytes_tlp(B, V, tail);
  if (!workspace_ok(workspace, workspace_bytes, need)) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_tlp(p, q1, q2, B, V, s, tail, r, omega1, w, accept, row_status, workspace,
                                   static_cast<hipStream_t>(stream)));
}

mdss_status mdss_select_truncated_lp(const float* p, const float* q1, const float* q2, const int32_t* drafts,
                                     const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t s,
                                     int32_t tail, const int32_t* omega1, const double* w, int32_t* sel_index,
                                     int32_t* sel_token, int32_t* row_status, void* stream) {
  if (tail != MDSS_TLP_SORTED && tail != MDSS_TLP_HALF) return MDSS_EINVAL;
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (s < 1 || s > MDSS_TLP_MAX_S) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q1 || !drafts || !omega1 || !w || !sel_index || !sel_token) return MDSS_EINVAL;
  return from_hip(mdss::launch_select_tlp(p, q1, q2, drafts, u, seed, offset, B, V, s, tail, omega1, w, sel_index,
                                          sel_token, row_status, static_cast<hipStream_t>(stream)));
}

size_t mdss_workspace_bytes_expsum(int64_t B, int64_t V, int32_t K) {
  if (check_shape(B, V) != MDSS_OK || K < 2 || K > MDSS_MAX_K || B == 0) return 0;
  return mdss::workspace_bytes_expsum(B, V, 1);
}

mdss_status mdss_induced_dist_expsum(const float* p, const float* q, int64_t B, int64_t V, int32_t K, float* r,
                                     int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r) return MDSS_EINVAL;
  if (!workspace_ok(workspace, workspace_bytes, mdss::workspace_bytes_expsum(B, V, 1))) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_expsum(p, q, nullptr, B, V, K, r, row_status, workspace,
                                              static_cast<hipStream_t>(stream)));
}

mdss_status mdss_induced_dist_topk_expsum(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                          int32_t s_max, float* r, int32_t* row_status, void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K || s_max < 1 || s_max > MDSS_K3_MAX_SUPPORT) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r) return MDSS_EINVAL;
  return from_hip(
      mdss::launch_induced_topk_expsum(p, q, B, V, K, s_max, r, row_status, static_cast<hipStream_t>(stream)));
}

mdss_status mdss_induced_dist_topk_expsum_sums(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                               int32_t s_max, float* r, int32_t* row_status, void* accept_workspace,
                                               size_t accept_workspace_bytes, void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K || s_max < 1 || s_max > MDSS_K3_MAX_SUPPORT) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r) return MDSS_EINVAL;
  if (!workspace_ok(accept_workspace, accept_workspace_bytes, mdss::workspace_bytes_accept(B, V)))
    return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_topk_expsum(p, q, B, V, K, s_max, r, row_status,
                                                   static_cast<hipStream_t>(stream),
                                                   static_cast<double*>(accept_workspace)));
}

mdss_status mdss_step_topk_expsum(const float* p, const float* q, const int32_t* drafts, const float* u,
                                  uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K, int32_t s_max,
                                  float* r, int32_t* sel_index, int32_t* sel_token, int32_t* out_token,
                                  uint8_t* accepted, double* residual_mass, int32_t* row_status,
                                  void* accept_workspace, size_t accept_workspace_bytes, void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K || s_max < 1 || s_max > MDSS_K3_MAX_SUPPORT) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r || !drafts || !out_token || !accepted) return MDSS_EINVAL;
  if (!workspace_ok(accept_workspace, accept_workspace_bytes, mdss::workspace_bytes_accept(B, V)))
    return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_step_topk_expsum(p, q, drafts, u, seed, offset, B, V, K, s_max, r, sel_index,
                                                sel_token, out_token, accepted, residual_mass, row_status,
                                                static_cast<double*>(accept_workspace),
                                                static_cast<hipStream_t>(stream)));
}

mdss_status mdss_induced_dist_expsum_noalloc(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                             float* r, int32_t* row_status, void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r) return MDSS_EINVAL;
  if (mdss::workspace_bytes_expsum(B, V, 1) > (size_t)MDSS_NOALLOC_SCRATCH_BYTES) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_expsum_noalloc(p, q, B, V, K, r, row_status, static_cast<hipStream_t>(stream)));
}

size_t mdss_workspace_bytes_pair_expsum(int64_t B, int64_t V) {
  if (check_shape(B, V) != MDSS_OK || B == 0) return 0;
  return mdss::workspace_bytes_expsum(B, V, 2);
}

mdss_status mdss_induced_dist_pair_expsum(const float* p, const float* q1, const float* q2, int64_t B, int64_t V,
                                          float* r, int32_t* row_status, void* workspace, size_t workspace_bytes,
                                          void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (B == 0) return MDSS_OK;
  if (!p || !q1 || !q2 || !r) return MDSS_EINVAL;
  if (!workspace_ok(workspace, workspace_bytes, mdss::workspace_bytes_expsum(B, V, 2))) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_expsum(p, q1, q2, B, V, 2, r, row_status, workspace,
                                              static_cast<hipStream_t>(stream)));
}

mdss_status mdss_induced_dist_successive_expsum(const float* p, const float* q, int64_t B, int64_t V, int32_t K,
                                                float* r_stages, int32_t* row_status, void* workspace,
                                                size_t workspace_bytes, void* stream) {
  const mdss_status st = check_shape(B, V);
  if (st != MDSS_OK) return st;
  if (K < 2 || K > MDSS_SUCCESSIVE_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r_stages) return MDSS_EINVAL;
  if (!workspace_ok(workspace, workspace_bytes, mdss::workspace_bytes_expsum(B, V, 2))) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_successive_expsum(p, q, B, V, K, r_stages, row_status, workspace,
                                                         static_cast<hipStream_t>(stream)));
}

mdss_status mdss_select_intermediate(const float* p, const float* q, const int32_t* drafts, const float* u,
                                     uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K,
                                     int32_t* sel_index, int32_t* sel_token, int32_t* row_status, void* stream) {
  mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !drafts || !sel_index || !sel_token) return MDSS_EINVAL;
  return from_hip(mdss::launch_select(p, q, drafts, u, seed, offset, B, V, K, sel_index, sel_token, row_status,
                                      static_cast<hipStream_t>(stream)));
}

size_t mdss_workspace_bytes_accept(int64_t B, int64_t V) {
  if (check_shape(B, V) != MDSS_OK || B == 0) return 0;
  return mdss::workspace_bytes_accept(B, V);
}

mdss_status mdss_accept_or_resample(const float* p, const float* r, const int32_t* sel_token, const float* u,
                                    uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t* out_token,
                                    uint8_t* accepted, float* residual, double* residual_mass, int32_t* row_status,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (B == 0) return MDSS_OK;
  if (!p || !r || !sel_token || !out_token || !accepted) return MDSS_EINVAL;
  if (!workspace_ok(workspace, workspace_bytes, mdss::workspace_bytes_accept(B, V))) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_accept(p, r, sel_token, u, seed, offset, B, V, out_token, accepted, residual,
                                      residual_mass, row_status, workspace, static_cast<hipStream_t>(stream)));
}

mdss_status mdss_select_accept(const float* p, const float* q, const float* r, const int32_t* drafts,
                               const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K,
                               int32_t* sel_index, int32_t* sel_token, int32_t* out_token, uint8_t* accepted,
                               float* residual, double* residual_mass, int32_t* row_status, void* workspace,
                               size_t workspace_bytes, void* stream) {
  mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r || !drafts || !out_token || !accepted) return MDSS_EINVAL;
  if (!workspace_ok(workspace, workspace_bytes, mdss::workspace_bytes_accept(B, V))) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_select_accept(p, q, nullptr, r, drafts, u, seed, offset, B, V, K, sel_index,
                                             sel_token, out_token, accepted, residual, residual_mass, row_status,
                                             workspace, static_cast<hipStream_t>(stream)));
}

mdss_status mdss_induced_dist_expsum_sums(const float* p, const float* q, int64_t B, int64_t V, int32_t K, float* r,
                                          int32_t* row_status, void* workspace, size_t workspace_bytes,
                                          void* accept_workspace, size_t accept_workspace_bytes, void* stream) {
  const mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r) return MDSS_EINVAL;
  if (!workspace_ok(workspace, workspace_bytes, mdss::workspace_bytes_expsum(B, V, 1))) return MDSS_EWORKSPACE;
  if (!workspace_ok(accept_workspace, accept_workspace_bytes, mdss::workspace_bytes_accept(B, V)))
    return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_induced_expsum(p, q, nullptr, B, V, K, r, row_status, workspace,
                                              static_cast<hipStream_t>(stream),
                                              static_cast<double*>(accept_workspace)));
}

mdss_status mdss_select_accept_sums(const float* p, const float* q, const float* r, const int32_t* drafts,
                                    const float* u, uint64_t seed, uint64_t offset, int64_t B, int64_t V, int32_t K,
                                    int32_t* sel_index, int32_t* sel_token, int32_t* out_token, uint8_t* accepted,
                                    double* residual_mass, int32_t* row_status, void* accept_workspace,
                                    size_t accept_workspace_bytes, void* stream) {
  mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (K < 2 || K > MDSS_MAX_K) return MDSS_EUNSUPPORTED;
  if (B == 0) return MDSS_OK;
  if (!p || !q || !r || !drafts || !out_token || !accepted) return MDSS_EINVAL;
  if (!workspace_ok(accept_workspace, accept_workspace_bytes, mdss::workspace_bytes_accept(B, V)))
    return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_select_accept_sums(p, q, nullptr, r, drafts, u, seed, offset, B, V, K, sel_index,
                                                  sel_token, out_token, accepted, residual_mass, row_status,
                                                  accept_workspace, static_cast<hipStream_t>(stream)));
}

mdss_status mdss_select_accept_pair(const float* p, const float* q1, const float* q2, const float* r,
                                    const int32_t* drafts, const float* u, uint64_t seed, uint64_t offset,
                                    int64_t B, int64_t V, int32_t* sel_index, int32_t* sel_token,
                                    int32_t* out_token, uint8_t* accepted, float* residual, double* residual_mass,
                                    int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream) {
  mdss_status s = check_shape(B, V);
  if (s != MDSS_OK) return s;
  if (B == 0) return MDSS_OK;
  if (!p || !q1 || !q2 || !r || !drafts || !out_token || !accepted) return MDSS_EINVAL;
  if (!workspace_ok(workspace, workspace_bytes, mdss::workspace_bytes_accept(B, V))) return MDSS_EWORKSPACE;
  return from_hip(mdss::launch_select_accept(p, q1, q2, r, drafts, u, seed, offset, B, V, 2, sel_index, sel_token,
                                             out_token, accepted, residual, residual_mass, row_status, workspace,
                                             static_cast<hipStream_t>(stream)));
}

}  // extern "C"
