/*
 * DO-loss reference oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct CPU implementation of what the DO-loss hot
 * path computes.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark may load it; the product library never does.  It
 * shares no code, header, table or helper with the HIP implementation.
 *
 * Paper: "Function Over Form: Distributional Orthogonalization in
 * Mixture-of-Experts with Replica Expert Mechanism" (arXiv 2609.32398).
 * Notation: the paper's m tokens / n experts / K selections are N / E / k here.
 *
 *   oracle_topk_signature  Sec. 3.1.1, Eq. (1): f_it = 1 iff expert i is among
 *                          the Top-K of token t.  Dense bool matrix F[E][N].
 *   oracle_pack            the binary load signature F_i as 64-bit words
 *                          (token t -> word t/64, bit t%64, tail bits 0).
 *   oracle_hamming         Eq. (6) magnitude term G_ij = ||F_i - F_j||_1,
 *                          computed from the definition as a count of
 *                          differing positions (not via the Gram identity).
 *   oracle_loss            Eq. (3): L_origin_DO = sum_{i != j} G_ij^2, with the
 *                          mean and population variance of the off-diagonal
 *                          distances (Sec. 3.1.1 / App. C.1: minimising the sum
 *                          of squares under the fixed total is minimising the
 *                          variance).  fp64 accumulation, plus exact u64 sums.
 *   oracle_surrogate       Sec. 3.1.3, Eq. (6)-(7): the surrogate loss
 *                          (1/(N^2 k)) sum_ij G_ij C_ij with the direction term
 *                          C_ij = sum_t p_it (f_it - f_jt) written out, and its
 *                          gradient with respect to the routing probabilities
 *                          p with G and F held constant.
 *   oracle_load_stats      per-expert loads n_i = ||F_i||_1 (App. C.3), the
 *                          Local-LBL balance loss sum_i f_i P_i of Sec. 4.2 and
 *                          the MaxVio imbalance of App. E over a placement of
 *                          the experts on ranks.
 *
 * Readings where the paper is silent:
 *   - ties in Top-K go to the lower expert index;
 *   - -0.0 equals +0.0 (IEEE comparison);
 *   - NaN ranks below every number including -inf, and all NaNs tie;
 *   - scores are ranked as given (no gating function is applied);
 *   - bf16 scores are widened exactly to fp32 (bits << 16) before comparing.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

typedef struct {
  uint64_t sum;   /* exact sum over i != j of D_ij */
  uint64_t sumsq; /* exact sum over i != j of D_ij^2 (Eq. 3) */
  double loss;    /* Eq. (3) accumulated in fp64 */
  double mean;    /* sum / (E(E-1)) */
  double var;     /* population variance of the off-diagonal D_ij, two-pass fp64 */
} oracle_loss_result;

static double score_at(const void* scores, int dtype, int64_t idx) {
  if (dtype == ORACLE_F32) return (double)((const float*)scores)[idx];
  uint32_t bits = (uint32_t)((const uint16_t*)scores)[idx] << 16;
  float f;
  memcpy(&f, &bits, 4);
  return (double)f;
}

/* Does expert a (value va) outrank expert b (value vb) for the same token? */
static int outranks(double va, int a, double vb, int b) {
  int na = isnan(va), nb = isnan(vb);
  if (na && nb) return a < b;
  if (na) return 0;
  if (nb) return 1;
  if (va > vb) return 1;
  if (va < vb) return 0;
  return a < b; /* equal values (this includes -0.0 == +0.0) */
}

/*
 * Eq. (1): for every token, pick k experts one at a time, each time the best
 * not yet chosen under `outranks`.  F must hold E*N bytes; F[e*N + t] is 0/1.
 */
int oracle_topk_signature(const void* scores, int dtype, int64_t N, int32_t E, int32_t k, uint8_t* F,
                          int nthreads) {
  if (N < 0 || E < 1 || k < 1 || k > E) return -1;
  memset(F, 0, (size_t)E * (size_t)N);
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : 1)
  {
    double* v = (double*)malloc(sizeof(double) * (size_t)E);
    uint8_t* chosen = (uint8_t*)malloc((size_t)E);
#pragma omp for schedule(static)
    for (int64_t t = 0; t < N; ++t) {
      for (int32_t e = 0; e < E; ++e) {
        v[e] = score_at(scores, dtype, t * E + e);
        chosen[e] = 0;
      }
      for (int32_t r = 0; r < k; ++r) {
        int32_t best = -1;
        for (int32_t e = 0; e < E; ++e) {
          if (chosen[e]) continue;
          if (best < 0 || outranks(v[e], e, v[best], best)) best = e;
        }
        chosen[best] = 1;
        F[(int64_t)best * N + t] = 1;
      }
    }
    free(v);
    free(chosen);
  }
  return 0;
}

/* Pack F[E][N] into words[E][ceil(N/64)]. */
int oracle_pack(const uint8_t* F, int64_t N, int32_t E, uint64_t* words) {
  int64_t W = (N + 63) / 64;
  memset(words, 0, sizeof(uint64_t) * (size_t)E * (size_t)W);
  for (int32_t e = 0; e < E; ++e)
    for (int64_t t = 0; t < N; ++t)
      if (F[(int64_t)e * N + t]) words[(int64_t)e * W + t / 64] |= (uint64_t)1 << (t % 64);
  return 0;
}

/* Eq. (6): D_ij = sum_t |f_it - f_jt| = number of tokens where exactly one of i, j is selected. */
int oracle_hamming(const uint8_t* F, int64_t N, int32_t E, uint32_t* D, int nthreads) {
  if (N < 0 || E < 1) return -1;
  int64_t npairs = (int64_t)E * E;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1)
  for (int64_t p = 0; p < npairs; ++p) {
    int32_t i = (int32_t)(p / E), j = (int32_t)(p % E);
    if (j < i) continue;
    const uint8_t* fi = F + (int64_t)i * N;
    const uint8_t* fj = F + (int64_t)j * N;
    uint64_t d = 0;
    for (int64_t t = 0; t < N; ++t) d += (uint64_t)(fi[t] != fj[t]);
    D[(int64_t)i * E + j] = (uint32_t)d;
    D[(int64_t)j * E + i] = (uint32_t)d;
  }
  return 0;
}

/* Eq. (3) and the statistics of the off-diagonal distances. */
int oracle_loss(const uint32_t* D, int32_t E, oracle_loss_result* out) {
  if (E < 1) return -1;
  memset(out, 0, sizeof(*out));
  if (E == 1) return 0;
  uint64_t s1 = 0, s2 = 0;
  double f2 = 0.0, f1 = 0.0;
  for (int32_t i = 0; i < E; ++i)
    for (int32_t j = 0; j < E; ++j) {
      if (i == j) continue;
      uint64_t d = D[(int64_t)i * E + j];
      s1 += d;
      s2 += d * d;
      f1 += (double)d;
      f2 += (double)d * (double)d;
    }
  double P = (double)E * (double)(E - 1);
  double mean = f1 / P;
  double acc = 0.0;
  for (int32_t i = 0; i < E; ++i)
    for (int32_t j = 0; j < E; ++j) {
      if (i == j) continue;
      double dev = (double)D[(int64_t)i * E + j] - mean;
      acc += dev * dev;
    }
  out->sum = s1;
  out->sumsq = s2;
  out->loss = f2;
  out->mean = mean;
  out->var = acc / P;
  return 0;
}

/*
 * Sec. 3.1.3, Eq. (6)-(7), surrogate loss with the magnitude G detached:
 *   C_ij = sum_t p_it (f_it - f_jt)
 *   L    = scale / (N^2 k) * sum_{i,j} G_ij C_ij
 *   dL/dp_it = scale / (N^2 k) * sum_j G_ij (f_it - f_jt)
 * p[N][E] (dtype as the scores), F[E][N] 0/1, G[E][E].  `scale` multiplies G
 * (1 on one device; Sec. 3.1.4 averages G over the data-parallel ranks).
 * grad (nullable) is [N][E].  Both quantities are evaluated from their
 * definitions, each with its own loop.
 */
int oracle_surrogate(const void* p, int dtype, int64_t N, int32_t E, int32_t k, const uint8_t* F, const uint32_t* G,
                     double scale, double* loss, double* grad, int nthreads) {
  if (N < 1 || E < 1 || k < 1 || k > E) return -1;
  const double norm = scale / ((double)N * (double)N * (double)k);
  double* C = (double*)calloc((size_t)E * (size_t)E, sizeof(double));
  if (!C) return -2;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1)
  for (int32_t i = 0; i < E; ++i)
    for (int32_t j = 0; j < E; ++j) {
      double c = 0.0;
      for (int64_t t = 0; t < N; ++t)
        c += score_at(p, dtype, t * E + i) * ((double)F[(int64_t)i * N + t] - (double)F[(int64_t)j * N + t]);
      C[(int64_t)i * E + j] = c;
    }
  double acc = 0.0;
  for (int32_t i = 0; i < E; ++i)
    for (int32_t j = 0; j < E; ++j) acc += (double)G[(int64_t)i * E + j] * C[(int64_t)i * E + j];
  *loss = norm * acc;
  free(C);
  if (grad) {
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t t = 0; t < N; ++t)
      for (int32_t i = 0; i < E; ++i) {
        double g = 0.0;
        for (int32_t j = 0; j < E; ++j)
          g += (double)G[(int64_t)i * E + j] * ((double)F[(int64_t)i * N + t] - (double)F[(int64_t)j * N + t]);
        grad[t * E + i] = norm * g;
      }
  }
  return 0;
}

/*
 * Load statistics of one layer's assignments F[E][N] (App. C.3, Sec. 4.2,
 * App. E).
 *   loads[i]  n_i = sum_t f_it, the number of tokens routed to expert i.
 *   lbl       Local-LBL sum_i f_i P_i with f_i = n_i / (N k), the fraction of
 *             the N k routing assignments that go to expert i, and
 *             P_i = (1/N) sum_t p_it, the mean routing probability; 0 when p
 *             is NULL.
 *   maxvio    max over ranks r of |L_r / tau - 1|, L_r the summed load of the
 *             experts placed on rank r (rank[i], R ranks; NULL: every expert
 *             its own rank), tau the mean of the L_r; 0 when tau is 0.
 * Returns -1 on bad arguments (including a rank outside [0, R)).
 */
typedef struct {
  uint64_t total;
  uint32_t max_load, min_load;
  double lbl;
  double maxvio;
} oracle_load_stats_result;

int oracle_load_stats(const uint8_t* F, int64_t N, int32_t E, int32_t k, const void* p, int dtype,
                      const int32_t* rank, int32_t R, uint32_t* loads, oracle_load_stats_result* out) {
  if (N < 1 || E < 1 || k < 1 || k > E) return -1;
  if (rank == NULL) R = E;
  if (R < 1) return -1;
  uint64_t total = 0;
  uint32_t mx = 0, mn = 0xFFFFFFFFu;
  for (int32_t i = 0; i < E; ++i) {
    uint64_t n = 0;
    for (int64_t t = 0; t < N; ++t) n += F[(int64_t)i * N + t];
    loads[i] = (uint32_t)n;
    total += n;
    if ((uint32_t)n > mx) mx = (uint32_t)n;
    if ((uint32_t)n < mn) mn = (uint32_t)n;
  }
  double lbl = 0.0;
  if (p != NULL) {
    for (int32_t i = 0; i < E; ++i) {
      double P = 0.0;
      for (int64_t t = 0; t < N; ++t) P += score_at(p, dtype, t * E + i);
      P /= (double)N;
      const double f = (double)loads[i] / ((double)N * (double)k);
      lbl += f * P;
    }
  }
  double* Lr = (double*)calloc((size_t)R, sizeof(double));
  if (!Lr) return -2;
  for (int32_t i = 0; i < E; ++i) {
    const int32_t r = rank ? rank[i] : i;
    if (r < 0 || r >= R) {
      free(Lr);
      return -1;
    }
    Lr[r] += (double)loads[i];
  }
  double tau = 0.0;
  for (int32_t r = 0; r < R; ++r) tau += Lr[r];
  tau /= (double)R;
  double mv = 0.0;
  if (tau > 0.0)
    for (int32_t r = 0; r < R; ++r) {
      const double v = fabs(Lr[r] / tau - 1.0);
      if (v > mv) mv = v;
    }
  free(Lr);
  out->total = total;
  out->max_load = mx;
  out->min_load = mn;
  out->lbl = lbl;
  out->maxvio = mv;
  return 0;
}
