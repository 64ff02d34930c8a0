/*
 * mdss_oracle.c -- plain fp64 CPU reference for multi-draft selection
 * (Khisti et al., "Multi-Draft Speculative Sampling: Canonical Decomposition
 * and Theoretical Limits", ICLR 2025).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  It shares no source with
 * the GPU library; the two never include or link each other.
 *
 * Notation: p = TARGET distribution, q = DRAFT distribution (the paper uses
 * the opposite letters).  w(x) = p(x)/q(x) is the classical importance
 * weight of a drafted token (Section 2, the remark after Definition 1).
 *
 * Everything is fp64, plain sequential loops, no fast-math and no floating
 * point contraction (built with -O2 -fno-fast-math -ffp-contract=off).
 * Inputs are fp32 arrays, promoted to fp64 on read, never renormalised.
 *
 * Row status bits (shared meaning with the public header, re-stated here):
 *   1  a probability in the row is NaN, infinite or negative
 *   2  a drafted / selected token id is out of range or has q = 0
 *   4  (GPU only: support larger than the caller's cap)
 *   8  rejection with zero residual mass: the selected token is output
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ST_BAD_PROB 1
#define ST_BAD_DRAFT 2
#define ST_FORCED 8

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 counter-based generator (Salmon, Moraes, Dror, Shaw,        */
/* "Parallel random numbers: as easy as 1, 2, 3", SC'11).  One round takes  */
/* the two 32x32->64 products of counter words 0 and 2 with the published   */
/* multipliers, swaps and xors the halves with the other counter words and  */
/* the round key; the key is advanced by the published Weyl increments      */
/* between rounds.                                                          */
/* ------------------------------------------------------------------------ */
void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint64_t prod0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
    uint64_t prod1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
    uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The three per-position uniforms: key = seed, counter = (position, 0, 0)
 * with the 64-bit position split low word first; output word j gives
 * u_j = (o_j >> 8) / 2^24, a 24-bit dyadic in [0,1). */
void oracle_uniforms(uint64_t seed, uint64_t position, float u[3]) {
  uint32_t ctr[4] = {(uint32_t)position, (uint32_t)(position >> 32), 0u, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t o[4];
  oracle_philox4x32_10(ctr, key, o);
  for (int j = 0; j < 3; ++j) u[j] = (float)((double)(o[j] >> 8) / 16777216.0);
}

/* ------------------------------------------------------------------------ */
/* helpers                                                                   */
/* ------------------------------------------------------------------------ */
static int bad_prob(float v) { return !(v >= 0.0f) || isinf(v); }

static int row_is_bad(const float* p, const float* q, int64_t V) {
  for (int64_t x = 0; x < V; ++x)
    if (bad_prob(p[x]) || bad_prob(q[x])) return 1;
  return 0;
}

/* Importance-sampling weights of one tuple of drafted tokens, index form:
 * Pr(I = i | x_1..x_K) = w(x_i) / sum_j w(x_j)  (the classical choice named
 * after Definition 1).  When every weight of the tuple is zero (all drafted
 * tokens have target probability 0) the ratio is 0/0; the reading taken is
 * the uniform choice 1/K over the indices. */
static void is_index_probs(const double* w_of_tuple, int K, double* beta) {
  double W = 0.0;
  for (int i = 0; i < K; ++i) W += w_of_tuple[i];
  for (int i = 0; i < K; ++i) beta[i] = (W > 0.0) ? w_of_tuple[i] / W : 1.0 / (double)K;
}

/* ------------------------------------------------------------------------ */
/* Induced distribution r = Pr(Y = y) of the importance-weighted selection. */
/* Definition 1 with the classical weights, marginalised over the drafts as */
/* in the first display of the proof of Theorem 1 (eq. Ind):               */
/*   r(y) = sum over ordered K-tuples x of prod_i q(x_i) * beta_y(x),       */
/* where beta_y(x) sums Pr(I = i | x) over the indices with x_i = y.  Only  */
/* tuples inside the support {q > 0} have non-zero probability, so the      */
/* enumeration runs over the support.                                       */
/* ------------------------------------------------------------------------ */
static void induced_row(const float* p, const float* q, int64_t V, int K, double* r) {
  int64_t n = 0;
  int64_t* supp = (int64_t*)malloc(sizeof(int64_t) * (size_t)(V > 0 ? V : 1));
  double* w = (double*)malloc(sizeof(double) * (size_t)(V > 0 ? V : 1));
  for (int64_t x = 0; x < V; ++x) {
    r[x] = 0.0;
    if (q[x] > 0.0f) {
      supp[n++] = x;
      w[x] = (double)p[x] / (double)q[x];
    }
  }
  if (n > 0) {
    int64_t idx[8] = {0};
    double wt[8], beta[8];
    for (;;) {
      double prob = 1.0;
      for (int i = 0; i < K; ++i) {
        int64_t x = supp[idx[i]];
        prob *= (double)q[x];
        wt[i] = w[x];
      }
      is_index_probs(wt, K, beta);
      for (int i = 0; i < K; ++i) r[supp[idx[i]]] += prob * beta[i];
      int d = K - 1; /* odometer over supp^K, last coordinate fastest */
      while (d >= 0 && ++idx[d] == n) idx[d--] = 0;
      if (d < 0) break;
    }
  }
  free(supp);
  free(w);
}

int oracle_induced_dist(const float* p, const float* q, int64_t B, int64_t V, int K, double* r, int32_t* status) {
  if (!p || !q || !r || B < 0 || V < 1 || K < 1 || K > 8) return 1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t b = 0; b < B; ++b) {
    const float* pb = p + b * V;
    const float* qb = q + b * V;
    double* rb = r + b * V;
    if (row_is_bad(pb, qb, V)) {
      for (int64_t x = 0; x < V; ++x) rb[x] = NAN;
      if (status) status[b] |= ST_BAD_PROB;
      continue;
    }
    induced_row(pb, qb, V, K, rb);
  }
  return 0;
}

/* One entry r(y) of row `row`, by the same definition restricted to the
 * tuples that contain y.  Those tuples are split by the first index j with
 * x_j = y (x_i != y for i < j, free for i > j), so every tuple is visited
 * once.  Cost K * n^(K-1) per entry instead of n^K per row. */
static double induced_entry(const float* p, const float* q, int64_t V, int K, int64_t y) {
  if (!(q[y] > 0.0f)) return 0.0;
  int64_t n = 0;
  int64_t* supp = (int64_t*)malloc(sizeof(int64_t) * (size_t)V);
  for (int64_t x = 0; x < V; ++x)
    if (q[x] > 0.0f) supp[n++] = x;
  double total = 0.0;
  int64_t x_t[8];
  double wt[8], beta[8];
  for (int j = 0; j < K; ++j) {
    /* free coordinates: all i != j; those before j must avoid y */
    int64_t idx[8] = {0};
    int nfree = K - 1;
    for (;;) {
      int ok = 1, f = 0;
      for (int i = 0; i < K; ++i) {
        if (i == j) { x_t[i] = y; continue; }
        x_t[i] = supp[idx[f++]];
        if (i < j && x_t[i] == y) ok = 0;
      }
      if (ok) {
        double prob = 1.0;
        for (int i = 0; i < K; ++i) {
          prob *= (double)q[x_t[i]];
          wt[i] = (double)p[x_t[i]] / (double)q[x_t[i]];
        }
        is_index_probs(wt, K, beta);
        double by = 0.0;
        for (int i = 0; i < K; ++i)
          if (x_t[i] == y) by += beta[i];
        total += prob * by;
      }
      if (nfree == 0) break;
      int d = nfree - 1;
      while (d >= 0 && ++idx[d] == n) idx[d--] = 0;
      if (d < 0) break;
    }
  }
  free(supp);
  return total;
}

int oracle_induced_dist_entries(const float* p, const float* q, int64_t V, int K, const int64_t* rows,
                                const int64_t* ys, int64_t count, double* out) {
  if (!p || !q || !rows || !ys || !out || V < 1 || K < 1 || K > 8) return 1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < count; ++i) {
    const float* pb = p + rows[i] * V;
    const float* qb = q + rows[i] * V;
    out[i] = row_is_bad(pb, qb, V) ? NAN : induced_entry(pb, qb, V, K, ys[i]);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Selection step (Definition 1, index form with the classical weights).    */
/* With W = sum_i w(x_i) and running sums C_i = w(x_1) + ... + w(x_i), the */
/* selected index is the smallest i with u_sel * W < C_i (inverse CDF of    */
/* the index distribution).  W = 0: index floor(u_sel * K).                 */
/* ------------------------------------------------------------------------ */
int oracle_select(const float* p, const float* q, const int32_t* drafts, const float* u, int64_t B, int64_t V, int K,
                  int32_t* sel_index, int32_t* sel_token, int32_t* status) {
  if (!p || !q || !drafts || !u || !sel_index || !sel_token || V < 1 || K < 1 || K > 8) return 1;
  for (int64_t b = 0; b < B; ++b) {
    const float* pb = p + b * V;
    const float* qb = q + b * V;
    int32_t st = 0;
    double w[8];
    for (int i = 0; i < K; ++i) {
      int32_t x = drafts[b * K + i];
      if (x < 0 || (int64_t)x >= V) { st |= ST_BAD_DRAFT; continue; }
      if (bad_prob(pb[x]) || bad_prob(qb[x])) { st |= ST_BAD_PROB; continue; }
      if (!(qb[x] > 0.0f)) { st |= ST_BAD_DRAFT; continue; }
      w[i] = (double)pb[x] / (double)qb[x];
    }
    if (st) {
      sel_index[b] = -1;
      sel_token[b] = -1;
      if (status) status[b] |= st;
      continue;
    }
    double W = 0.0;
    for (int i = 0; i < K; ++i) W += w[i];
    double us = (double)u[b * 3 + 0];
    int istar = K - 1;
    if (W > 0.0) {
      double t = us * W, C = 0.0;
      for (int i = 0; i < K; ++i) {
        C += w[i];
        if (t < C) { istar = i; break; }
      }
    } else {
      istar = (int)floor(us * (double)K);
    }
    sel_index[b] = istar;
    sel_token[b] = drafts[b * K + istar];
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Single-draft speculative sampling of the selected token against the      */
/* target (Algorithm 1 in the speculative-sampling appendix, with the      */
/* induced distribution r in the role of the draft):                        */
/*   accept with probability min(1, p(Y)/r(Y)): accept iff u_acc r(Y) < p(Y) */
/*   (exact in fp64: both factors carry at most 24 significant bits);        */
/*   otherwise draw from the residual res(x) = max(0, p(x) - r(x)) divided  */
/*   by its mass Z: the smallest token j with C_j > u_res * Z, C_j the      */
/*   running sum of res in ascending token id.                              */
/* Z = 0 on a rejection (only possible when the fp32 rows do not carry equal */
/* mass): the selected token is output and status bit 8 is set.            */
/* residual (nullable) receives res for every row; mass (nullable) Z.       */
/* ------------------------------------------------------------------------ */
int oracle_accept_resample(const float* p, const float* r, const int32_t* sel_token, const float* u, int64_t B,
                           int64_t V, int32_t* out_token, uint8_t* accepted, double* residual, double* mass,
                           int32_t* status) {
  if (!p || !r || !sel_token || !u || !out_token || !accepted || V < 1) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < B; ++b) {
    const float* pb = p + b * V;
    const float* rb = r + b * V;
    int32_t Y = sel_token[b];
    double Z = 0.0;
    int bad = 0;
    for (int64_t x = 0; x < V; ++x) {
      if (bad_prob(pb[x]) || bad_prob(rb[x])) bad = 1;
      double d = (double)pb[x] - (double)rb[x];
      double res = d > 0.0 ? d : 0.0;
      if (residual) residual[b * V + x] = res;
      Z += res;
    }
    if (mass) mass[b] = bad ? NAN : Z;
    if (bad || Y < 0 || (int64_t)Y >= V) {
      out_token[b] = -1;
      accepted[b] = 0;
      if (status) status[b] |= bad ? ST_BAD_PROB : ST_BAD_DRAFT;
      continue;
    }
    double ua = (double)u[b * 3 + 1], ur = (double)u[b * 3 + 2];
    if (ua * (double)rb[Y] < (double)pb[Y]) {
      out_token[b] = Y;
      accepted[b] = 1;
      continue;
    }
    if (!(Z > 0.0)) {
      out_token[b] = Y;
      accepted[b] = 1;
      if (status) status[b] |= ST_FORCED;
      continue;
    }
    double t = ur * Z, C = 0.0;
    int32_t z = -1;
    for (int64_t x = 0; x < V; ++x) {
      double d = (double)pb[x] - (double)rb[x];
      C += d > 0.0 ? d : 0.0;
      if (C > t) { z = (int32_t)x; break; }
    }
    out_token[b] = z;
    accepted[b] = 0;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Two drafts from different distributions (Remark 1; the non-identical     */
/* K = 2 appendix): X1 ~ q1, X2 ~ q2 independent.  The classical weight of */
/* draft i is w_i(x) = p(x)/q_i(x) (target over the distribution that      */
/* proposed it); Pr(I = i | x1, x2) = w_i(x_i) / (w_1(x1) + w_2(x2)), the   */
/* uniform choice when both are zero.  r(y) sums q1(x1) q2(x2) times the    */
/* probability of selecting y over all ordered pairs of the two supports.   */
/* ------------------------------------------------------------------------ */
static void induced_pair_row(const float* p, const float* q1, const float* q2, int64_t V, double* r) {
  int64_t n1 = 0, n2 = 0;
  int64_t* s1 = (int64_t*)malloc(sizeof(int64_t) * (size_t)V);
  int64_t* s2 = (int64_t*)malloc(sizeof(int64_t) * (size_t)V);
  for (int64_t x = 0; x < V; ++x) {
    r[x] = 0.0;
    if (q1[x] > 0.0f) s1[n1++] = x;
    if (q2[x] > 0.0f) s2[n2++] = x;
  }
  double wt[2], beta[2];
  for (int64_t i = 0; i < n1; ++i) {
    const int64_t x1 = s1[i];
    for (int64_t j = 0; j < n2; ++j) {
      const int64_t x2 = s2[j];
      const double prob = (double)q1[x1] * (double)q2[x2];
      wt[0] = (double)p[x1] / (double)q1[x1];
      wt[1] = (double)p[x2] / (double)q2[x2];
      is_index_probs(wt, 2, beta);
      r[x1] += prob * beta[0];
      r[x2] += prob * beta[1];
    }
  }
  free(s1);
  free(s2);
}

int oracle_induced_dist_pair(const float* p, const float* q1, const float* q2, int64_t B, int64_t V, double* r,
                             int32_t* status) {
  if (!p || !q1 || !q2 || !r || B < 0 || V < 1) return 1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t b = 0; b < B; ++b) {
    const float* pb = p + b * V;
    const float* q1b = q1 + b * V;
    const float* q2b = q2 + b * V;
    double* rb = r + b * V;
    if (row_is_bad(pb, q1b, V) || row_is_bad(pb, q2b, V)) {
      for (int64_t x = 0; x < V; ++x) rb[x] = NAN;
      if (status) status[b] |= ST_BAD_PROB;
      continue;
    }
    induced_pair_row(pb, q1b, q2b, V, rb);
  }
  return 0;
}

/* One entry r(y) of the two-draft distribution, from the pairs with x1 = y or x2 = y. */
int oracle_induced_dist_pair_entries(const float* p, const float* q1, const float* q2, int64_t V, const int64_t* rows,
                                     const int64_t* ys, int64_t count, double* out) {
  if (!p || !q1 || !q2 || !rows || !ys || !out || V < 1) return 1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < count; ++i) {
    const float* pb = p + rows[i] * V;
    const float* q1b = q1 + rows[i] * V;
    const float* q2b = q2 + rows[i] * V;
    const int64_t y = ys[i];
    if (row_is_bad(pb, q1b, V) || row_is_bad(pb, q2b, V)) {
      out[i] = NAN;
      continue;
    }
    double total = 0.0, wt[2], beta[2];
    /* pairs (y, x2) for every x2, then (x1, y) for x1 != y */
    for (int pass = 0; pass < 2; ++pass) {
      for (int64_t x = 0; x < V; ++x) {
        const int64_t x1 = pass == 0 ? y : x, x2 = pass == 0 ? x : y;
        if (pass == 1 && x == y) continue;
        if (!(q1b[x1] > 0.0f) || !(q2b[x2] > 0.0f)) continue;
        const double prob = (double)q1b[x1] * (double)q2b[x2];
        wt[0] = (double)pb[x1] / (double)q1b[x1];
        wt[1] = (double)pb[x2] / (double)q2b[x2];
        is_index_probs(wt, 2, beta);
        total += prob * ((x1 == y ? beta[0] : 0.0) + (x2 == y ? beta[1] : 0.0));
      }
    }
    out[i] = total;
  }
  return 0;
}

/* Selection between two drafts proposed by different distributions:
 * w_1 = p(x1)/q1(x1), w_2 = p(x2)/q2(x2), then the same inverse CDF as
 * oracle_select (index 0 iff u * W < w_1; W = 0: floor(2 u)). */
int oracle_select_pair(const float* p, const float* q1, const float* q2, const int32_t* drafts, const float* u,
                       int64_t B, int64_t V, int32_t* sel_index, int32_t* sel_token, int32_t* status) {
  if (!p || !q1 || !q2 || !drafts || !u || !sel_index || !sel_token || V < 1) return 1;
  for (int64_t b = 0; b < B; ++b) {
    const float* pb = p + b * V;
    const float* qs[2] = {q1 + b * V, q2 + b * V};
    int32_t st = 0;
    double w[2] = {0.0, 0.0};
    for (int i = 0; i < 2; ++i) {
      int32_t x = drafts[b * 2 + i];
      if (x < 0 || (int64_t)x >= V) { st |= ST_BAD_DRAFT; continue; }
      if (bad_prob(pb[x]) || bad_prob(qs[i][x])) { st |= ST_BAD_PROB; continue; }
      if (!(qs[i][x] > 0.0f)) { st |= ST_BAD_DRAFT; continue; }
      w[i] = (double)pb[x] / (double)qs[i][x];
    }
    if (st) {
      sel_index[b] = -1;
      sel_token[b] = -1;
      if (status) status[b] |= st;
      continue;
    }
    const double W = w[0] + w[1];
    const double us = (double)u[b * 3 + 0];
    int istar;
    if (W > 0.0) {
      istar = (us * W < w[0]) ? 0 : 1;
    } else {
      istar = (int)floor(us * 2.0);
    }
    sel_index[b] = istar;
    sel_token[b] = drafts[b * 2 + istar];
  }
  return 0;
}
