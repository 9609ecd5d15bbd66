/*
 * Seeded synthetic router-score generator.
 *
 * Shared by the test/bench harness on both sides of every parity check (the
 * CPU oracle and the HIP path consume the very same bytes).  It holds no
 * DO-loss arithmetic: it only draws counter-based random numbers and shapes
 * them into the score distributions of the synthetic workloads.
 *
 * Random numbers: SplitMix64-style finaliser applied to a counter derived from
 * (seed, stream, index), so any token range of any layer can be generated
 * independently and in parallel.  Normals: Box-Muller in fp64 on a pair of
 * uniforms; the pair index is (token*E + expert) / 2, the even member takes
 * the cosine branch and the odd member the sine branch.
 *
 * Rounding: fp64 -> fp32 by C conversion (round to nearest even), fp32 ->
 * bf16 by round-to-nearest-even on the bit pattern.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SYNTH_F32 0
#define SYNTH_BF16 1

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
  return mix64(mix64(seed + 0x632BE59BD9B4E019ULL) ^ (stream * 0x9E3779B97F4A7C15ULL + 0xD1B54A32D192ED03ULL));
}

static inline uint64_t ctr(uint64_t key, uint64_t i) {
  return mix64(key + (i + 1) * 0x9E3779B97F4A7C15ULL);
}

/* uniform in (0, 1), never 0 */
static inline double u01(uint64_t r) { return ((double)(r >> 11) + 0.5) * (1.0 / 9007199254740992.0); }

/* standard normal number `i` of the stream with key `key` */
static inline double normal_at(uint64_t key, uint64_t i) {
  uint64_t p = i >> 1;
  double u1 = u01(ctr(key, 2 * p));
  double u2 = u01(ctr(key, 2 * p + 1));
  double r = sqrt(-2.0 * log(u1));
  double th = 6.283185307179586476925286766559 * u2;
  return (i & 1) ? r * sin(th) : r * cos(th);
}


/* Fill dst[0..cnt) with normals number i0, i0+1, ... of the stream (pair-wise Box-Muller). */
static void normals_fill(uint64_t key, uint64_t i0, int64_t cnt, double* dst) {
  int64_t j = 0;
  if ((i0 & 1) && cnt > 0) { dst[0] = normal_at(key, i0); j = 1; }
  while (j + 1 < cnt) {
    double u1[128], u2[128], r[128], c[128], s[128];
    int64_t np = (cnt - j) / 2;
    if (np > 128) np = 128;
    uint64_t p0 = (i0 + (uint64_t)j) >> 1;
    for (int64_t q = 0; q < np; ++q) {
      u1[q] = u01(ctr(key, 2 * (p0 + (uint64_t)q)));
      u2[q] = 6.283185307179586476925286766559 * u01(ctr(key, 2 * (p0 + (uint64_t)q) + 1));
    }
#pragma omp simd
    for (int64_t q = 0; q < np; ++q) {
      r[q] = sqrt(-2.0 * log(u1[q]));
      c[q] = cos(u2[q]);
      s[q] = sin(u2[q]);
    }
    for (int64_t q = 0; q < np; ++q) {
      dst[j + 2 * q] = r[q] * c[q];
      dst[j + 2 * q + 1] = r[q] * s[q];
    }
    j += 2 * np;
  }
  if (j < cnt) dst[j] = normal_at(key, i0 + (uint64_t)j);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40); /* quiet NaN */
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline void store(void* out, int dtype, int64_t idx, double v) {
  float f = (float)v;
  if (dtype == SYNTH_F32)
    ((float*)out)[idx] = f;
  else
    ((uint16_t*)out)[idx] = f32_to_bf16_rne(f);
}

/* ---------------------------------------------------------------------------
 * Generic generators used by the tests.
 * ------------------------------------------------------------------------- */

/* out[n][E] = mean + std * N(0,1), tokens are rows [t0, t0+n) of stream `stream` */
int synth_normal(uint64_t seed, uint64_t stream, int dtype, int64_t t0, int64_t n, int32_t E,
                 double mean, double std, void* out, int nthreads) {
  if (n < 0 || E < 1 || (dtype != SYNTH_F32 && dtype != SYNTH_BF16)) return -1;
  uint64_t key = stream_key(seed, stream);
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
  for (int64_t t = 0; t < n; ++t) {
    double z[4096];
    for (int32_t e0 = 0; e0 < E; e0 += 4096) {
      int32_t m = E - e0 < 4096 ? E - e0 : 4096;
      normals_fill(key, (uint64_t)(t0 + t) * (uint64_t)E + (uint64_t)e0, m, z);
      for (int32_t e = 0; e < m; ++e) store(out, dtype, t * E + e0 + e, mean + std * z[e]);
    }
  }
  return 0;
}

/* Tie-heavy integer-valued scores drawn uniformly from [lo, hi]. */
int synth_int_ties(uint64_t seed, uint64_t stream, int dtype, int64_t n, int32_t E, int32_t lo, int32_t hi,
                   void* out, int nthreads) {
  if (n < 0 || E < 1 || hi < lo) return -1;
  uint64_t key = stream_key(seed, stream);
  uint64_t span = (uint64_t)(hi - lo) + 1;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : 1)
  for (int64_t t = 0; t < n; ++t)
    for (int32_t e = 0; e < E; ++e) {
      uint64_t i = (uint64_t)t * (uint64_t)E + (uint64_t)e;
      store(out, dtype, t * E + e, (double)(lo + (int64_t)(ctr(key, i) % span)));
    }
  return 0;
}

/* ---------------------------------------------------------------------------
 * The five synthetic workloads.
 *
 *  0: fp32, 1 layer,  N=4096,   E=8,   k=2; N(0,1) i.i.d.
 *  1: bf16, 1 layer,  N=65536,  E=64,  k=6; N(0,1) + per-expert bias b_e ~ N(0, 0.5^2)
 *  2: bf16, 48 layers, N=262144, E=128, k=8; N(0,1), 16 experts per layer biased by -10
 *  3: bf16, 16 micro-batches of 65536 tokens, E=128, k=8; N(0,1) - 1.1*ln(r_e),
 *     r_e a seeded permutation of 1..128 (Zipf-like popularity), same bias for
 *     every micro-batch; "layer" selects the micro-batch
 *  4: fp32, 8 layers, N=4194304, E=256, k=8; per-token softmax (fp64) of
 *     N(0,1) + 2.0 * [expert favoured by the token's cluster]; 32 clusters per
 *     layer, each favouring 8 distinct experts; clusters drawn uniformly
 * ------------------------------------------------------------------------- */

#define SYNTH_BASE_SEED 0x32398ULL

typedef struct {
  int64_t layers, n, E, k, dtype;
} cfg_shape;

static const cfg_shape CFG[5] = {
    {1, 4096, 8, 2, SYNTH_F32},
    {1, 65536, 64, 6, SYNTH_BF16},
    {48, 262144, 128, 8, SYNTH_BF16},
    {16, 65536, 128, 8, SYNTH_BF16},
    {8, 4194304, 256, 8, SYNTH_F32},
};

int synth_config_shape(int cfg, int64_t* layers, int64_t* n, int32_t* E, int32_t* k, int32_t* dtype) {
  if (cfg < 0 || cfg > 4) return -1;
  *layers = CFG[cfg].layers;
  *n = CFG[cfg].n;
  *E = (int32_t)CFG[cfg].E;
  *k = (int32_t)CFG[cfg].k;
  *dtype = (int32_t)CFG[cfg].dtype;
  return 0;
}

/* distinct picks: the first m entries of a seeded Fisher-Yates shuffle of 0..E-1 */
static void shuffle_prefix(uint64_t key, int32_t E, int32_t m, int32_t* out) {
  int32_t* perm = (int32_t*)malloc(sizeof(int32_t) * (size_t)E);
  for (int32_t i = 0; i < E; ++i) perm[i] = i;
  for (int32_t i = 0; i < m && i < E - 1; ++i) {
    int32_t j = i + (int32_t)(ctr(key, (uint64_t)i) % (uint64_t)(E - i));
    int32_t t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
  for (int32_t i = 0; i < m; ++i) out[i] = perm[i];
  free(perm);
}

/* Per-expert bias of workloads 1-3 (zero where the workload has none). */
int synth_config_bias(int cfg, int layer, double* bias) {
  if (cfg < 0 || cfg > 4) return -1;
  int32_t E = (int32_t)CFG[cfg].E;
  uint64_t seed = SYNTH_BASE_SEED + (uint64_t)cfg;
  for (int32_t e = 0; e < E; ++e) bias[e] = 0.0;
  if (cfg == 1) {
    uint64_t key = stream_key(seed, 1000003);
    for (int32_t e = 0; e < E; ++e) bias[e] = 0.5 * normal_at(key, (uint64_t)e);
  } else if (cfg == 2) {
    int32_t idle[16];
    shuffle_prefix(stream_key(seed, 2000000 + (uint64_t)layer), E, 16, idle);
    for (int i = 0; i < 16; ++i) bias[idle[i]] = -10.0;
  } else if (cfg == 3) {
    int32_t* perm = (int32_t*)malloc(sizeof(int32_t) * (size_t)E);
    shuffle_prefix(stream_key(seed, 3000000), E, E, perm);
    /* expert perm[r-1] has popularity rank r */
    for (int32_t r = 1; r <= E; ++r) bias[perm[r - 1]] = -1.1 * log((double)r);
    free(perm);
  }
  return 0;
}

/* favoured experts of workload 4: fav[32][8] for the given layer */
int synth_config_clusters(int layer, int32_t* fav) {
  uint64_t seed = SYNTH_BASE_SEED + 4;
  for (int c = 0; c < 32; ++c)
    shuffle_prefix(stream_key(seed, 4000000 + (uint64_t)layer * 64 + (uint64_t)c), 256, 8, fav + c * 8);
  return 0;
}

int synth_config_fill(int cfg, int layer, int64_t t0, int64_t n, void* out, int nthreads) {
  if (cfg < 0 || cfg > 4) return -1;
  const cfg_shape s = CFG[cfg];
  if (layer < 0 || layer >= s.layers || t0 < 0 || n < 0 || t0 + n > s.n) return -1;
  int32_t E = (int32_t)s.E;
  int dtype = (int)s.dtype;
  uint64_t seed = SYNTH_BASE_SEED + (uint64_t)cfg;
  uint64_t key = stream_key(seed, (uint64_t)layer);
  int nt = nthreads > 0 ? nthreads : 1;
  if (cfg <= 3) {
    double bias[256];
    synth_config_bias(cfg, layer, bias);
#pragma omp parallel for schedule(static) num_threads(nt)
    for (int64_t t = 0; t < n; ++t) {
      double z[256];
      normals_fill(key, (uint64_t)(t0 + t) * (uint64_t)E, E, z);
      for (int32_t e = 0; e < E; ++e) store(out, dtype, t * E + e, z[e] + bias[e]);
    }
    return 0;
  }
  /* workload 4 */
  int32_t fav[32 * 8];
  synth_config_clusters(layer, fav);
  uint64_t ckey = stream_key(seed, 5000000 + (uint64_t)layer);
#pragma omp parallel for schedule(static) num_threads(nt)
  for (int64_t t = 0; t < n; ++t) {
    double logit[256];
    int64_t tok = t0 + t;
    int c = (int)(ctr(ckey, (uint64_t)tok) % 32u);
    normals_fill(key, (uint64_t)tok * (uint64_t)E, E, logit);
    for (int j = 0; j < 8; ++j) logit[fav[c * 8 + j]] += 2.0;
    double m = logit[0];
    for (int32_t e = 1; e < E; ++e) m = logit[e] > m ? logit[e] : m;
    double z = 0.0;
#pragma omp simd
    for (int32_t e = 0; e < E; ++e) logit[e] = exp(logit[e] - m);
    for (int32_t e = 0; e < E; ++e) z += logit[e];
    for (int32_t e = 0; e < E; ++e) store(out, dtype, t * E + e, logit[e] / z);
  }
  return 0;
}
