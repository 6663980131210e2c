/*
 * QuantWM CPU oracle: TEST INFRASTRUCTURE ONLY (see quantwm_oracle.h).
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fopenmp -shared -fPIC.
 * Contraction stays off so that every a*b+c below is two roundings.
 *
 * Readings of the paper that this file takes:
 *  - The quantiser range is extended to contain 0, so the INT2 zero-point always
 *    lies in [0, 3] and can be bit-packed (Eq. 2 with App. D.1).
 *  - The residual is quantised with the stored (FP16-rounded) scale.
 *  - A group whose stored scale is 0 keeps all codes 0 (reconstruction = centroid).
 *  - Eq. 10's range R_g is the literal max - min, without the 0 extension.
 *  - Ties: the lower centroid id wins; eigenvalue ties keep the original order;
 *    each eigenvector's largest-magnitude entry is made positive.
 *  - Values take the nearest centroid (w = 1, M = 1) and no PSAC (App. D.1).
 *  - PSAC coefficients are INT8, symmetric, one FP16 scale per row (max|C|/127).
 *  - Cold start (no historical Queries): w = 1 and U_r = 0, so PSAC stores zero
 *    rows (App. C.3).
 *  - K-means: Lloyd on the calibration tokens, initial centroids at tokens
 *    floor(i*N/Kc), empty clusters keep their centroid, centroids are rounded to
 *    the table type after every update.
 */
#include "quantwm_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- formats */

/* Round to a binary format with p significand bits (hidden bit included) whose
 * smallest normal exponent is emin; below it the spacing stays 2^(emin-p+1). */
static double round_format(double x, int p, int emin) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  frexp(x, &e); /* |x| in [2^(e-1), 2^e) */
  int lsb = (e - 1) - (p - 1);
  if (lsb < emin - (p - 1)) lsb = emin - (p - 1);
  return ldexp(nearbyint(ldexp(x, -lsb)), lsb); /* default mode: ties to even */
}

double ora_round_bf16(double x) { return round_format(x, 8, -126); }

double ora_round_f16(double x) {
  double r = round_format(x, 11, -14);
  if (fabs(r) > 65504.0) r = copysign(INFINITY, r);
  return r;
}

static double round_f32(double x) { return (double)(float)x; }

static double round_table(const ora_cfg* c, double x) {
  return c->table_bf16 ? ora_round_bf16(x) : round_f32(x);
}

uint16_t ora_f16_bits(double v) {
  uint16_t s = signbit(v) ? 0x8000u : 0u;
  double a = fabs(v);
  if (a == 0.0) return s;
  if (isinf(a)) return (uint16_t)(s | 0x7C00u);
  if (a < ldexp(1.0, -14)) return (uint16_t)(s | (uint16_t)ldexp(a, 24)); /* subnormal */
  int e;
  frexp(a, &e);
  int exp_field = (e - 1) + 15;
  int mant = (int)(ldexp(a, -(e - 1)) * 1024.0) - 1024;
  return (uint16_t)(s | (exp_field << 10) | mant);
}

double ora_f16_value(uint16_t bits) {
  int s = bits >> 15, ef = (bits >> 10) & 31, m = bits & 1023;
  double v;
  if (ef == 0) v = ldexp((double)m, -24);
  else if (ef == 31) v = m ? NAN : INFINITY;
  else v = ldexp((double)(1024 + m), ef - 15 - 10);
  return s ? -v : v;
}

/* ----------------------------------------------------------------- layout */

typedef struct {
  int d, ng, zpb, r;
  int k_bytes, v_bytes;
  long long slots; /* capacity rounded up to 64 */
  int i8;            /* ORA_STORE_SCALE_I8 */
  int sb;            /* group-scale bytes per token: 2 ng (FP16) or ng (8-bit codes) */
  long long k_codes, k_ids, k_zp, k_scale, k_coef, k_cscale;
  long long v_codes, v_ids, v_zp, v_scale;
  long long k_sigma, v_sigma; /* SCALE_I8: the FP16 secondary scale per token */
  int sparse;                 /* SPARSE: rows in a pool with a tile directory */
  long long pool;             /* rows per (b, h) in the coefficient sections */
  long long k_dir, k_over;    /* SPARSE: directory and overflow counters */
  long long stage;            /* SPARSE: staging rows per (b, h) */
  long long k_st_codes, k_st_scale;
  long long total;
} layout;

static long long up256(long long x) { return (x + 255) / 256 * 256; }

/* head_dim is at most 256: the per-token buffers below are sized for it. */
static int valid_cfg(const ora_cfg* c) {
  if (!c || c->batch < 1 || c->heads < 1 || c->head_dim < 4 || c->head_dim % 4 || c->head_dim > 256) return 0;
  if (c->group_size < 1 || c->head_dim % c->group_size) return 0;
  if (c->n_centroids < 1 || c->n_centroids > 256) return 0;
  if (c->rank < 0 || c->rank > c->head_dim) return 0;
  if (c->top_m < 1 || c->capacity < 0) return 0;
  if (c->storage & ~(ORA_STORE_SCALE_I8 | ORA_STORE_GATE | ORA_STORE_SPARSE)) return 0;
  if ((c->storage & ORA_STORE_SPARSE) && (c->rank < 1 || c->coef_rows < 0 || c->coef_stage < 1)) return 0;
  if (c->metric != ORA_METRIC_DIAG && c->metric != ORA_METRIC_FULL) return 0;
  return 1;
}

static layout make_layout(const ora_cfg* c) {
  layout L;
  L.d = c->head_dim;
  L.ng = c->head_dim / c->group_size;
  L.zpb = (L.ng + 3) / 4;
  L.r = c->rank;
  L.slots = (c->capacity + 63) / 64 * 64;
  L.i8 = (c->storage & ORA_STORE_SCALE_I8) != 0;
  L.sb = L.i8 ? L.ng : 2 * L.ng;
  L.sparse = (c->storage & ORA_STORE_SPARSE) != 0;
  L.pool = L.sparse && c->coef_rows > 0 ? c->coef_rows : L.slots;
  long long bh = (long long)c->batch * c->heads, n = bh * L.slots, off = 0;
#define SECTION_N(field, rows, per_row) \
  do { L.field = off; off = up256(off + (rows) * (long long)(per_row)); } while (0)
#define SECTION(field, per_token) SECTION_N(field, n, per_token)
  SECTION(k_codes, L.d / 4);
  SECTION(k_ids, 1);
  SECTION(k_zp, L.zpb);
  SECTION(k_scale, L.sb);
  SECTION_N(k_coef, bh * L.pool, L.r);
  SECTION_N(k_cscale, bh * L.pool, L.r > 0 ? 2 : 0);
  SECTION(v_codes, L.d / 4);
  SECTION(v_ids, 1);
  SECTION(v_zp, L.zpb);
  SECTION(v_scale, L.sb);
  SECTION(k_sigma, L.i8 ? 2 : 0);
  SECTION(v_sigma, L.i8 ? 2 : 0);
  SECTION_N(k_dir, bh * (L.slots / 64), L.sparse ? 16 : 0);
  SECTION_N(k_over, bh, L.sparse ? 4 : 0);
  L.stage = L.sparse ? c->coef_stage : 0;
  SECTION_N(k_st_codes, bh * L.stage, L.r);
  SECTION_N(k_st_scale, bh * L.stage, 2);
#undef SECTION
#undef SECTION_N
  L.total = off;
  L.v_bytes = L.d / 4 + 1 + L.zpb + L.sb + (L.i8 ? 2 : 0);
  L.k_bytes = L.v_bytes + (L.r > 0 ? L.r + 2 : 0);
  return L;
}

long long ora_cache_bytes(const ora_cfg* cfg) {
  if (!valid_cfg(cfg)) return -1;
  return make_layout(cfg).total;
}

int ora_token_bytes(const ora_cfg* cfg, int* k_bytes, int* v_bytes) {
  if (!valid_cfg(cfg)) return -1;
  layout L = make_layout(cfg);
  *k_bytes = L.k_bytes;
  *v_bytes = L.v_bytes;
  return 0;
}

static void put16(uint8_t* p, uint16_t v) { p[0] = (uint8_t)(v & 255); p[1] = (uint8_t)(v >> 8); }
static uint16_t get16(const uint8_t* p) { return (uint16_t)(p[0] | (p[1] << 8)); }
static void put32(uint8_t* p, uint32_t v) {
  for (int i = 0; i < 4; ++i) p[i] = (uint8_t)(v >> (8 * i));
}
static uint32_t get32(const uint8_t* p) {
  return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}
static uint64_t get64(const uint8_t* p) { return (uint64_t)get32(p) | ((uint64_t)get32(p + 4) << 32); }
static void put64(uint8_t* p, uint64_t v) { put32(p, (uint32_t)v); put32(p + 4, (uint32_t)(v >> 32)); }
static int popcount64(uint64_t x) {
  int c = 0;
  for (; x; x &= x - 1) ++c;
  return c;
}

/* ------------------------------------------- resident sparse PSAC rows */

/* Directory entry of tile T of head bh: {u32 base, u32 0, u64 mask}. */
static uint8_t* dir_entry(const layout* L, uint8_t* cache, long long bh, long long T) {
  return cache + L->k_dir + (bh * (L->slots / 64) + T) * 16;
}

/* Pool rows used by the slots below `slot` of head bh (the rows are stored in
 * slot order, so this is where the next row goes). */
static long long pool_fill(const layout* L, const uint8_t* cache, long long bh, long long slot) {
  if (slot == 0) return 0;
  const long long T = (slot - 1) / 64;
  const uint8_t* e = cache + L->k_dir + (bh * (L->slots / 64) + T) * 16;
  const int used = (int)(slot - 64 * T); /* slots of tile T below `slot`: 1..64 */
  const uint64_t below = used == 64 ? ~(uint64_t)0 : (((uint64_t)1 << used) - 1);
  return (long long)get32(e) + popcount64(get64(e + 8) & below);
}

/* Pool row of slot t of head bh, or -1 when the slot has none. */
static long long pool_row(const layout* L, const uint8_t* cache, long long bh, long long t) {
  const uint8_t* e = cache + L->k_dir + (bh * (L->slots / 64) + t / 64) * 16;
  const int i = (int)(t % 64);
  const uint64_t mask = get64(e + 8);
  if (!((mask >> i) & 1)) return -1;
  return (long long)get32(e) + popcount64(mask & (((uint64_t)1 << i) - 1));
}

/* Stores one append call's rows of head bh, staged in the cache (for slots
 * [n_cached, n_cached + n)), into the pool: the whole chunk (dense) or its
 * non-zero-scale rows (sparse), whichever is smaller with one mask bit per slot
 * as the sparse index (ties dense); then the directory of its tiles. */
static void sparse_commit(const layout* L, uint8_t* cache, long long bh, long long n_cached, long long n) {
  const int r = L->r;
  const int8_t* codes = (const int8_t*)(cache + L->k_st_codes + bh * L->stage * r);
  const uint8_t* sb = cache + L->k_st_scale + bh * L->stage * 2;
  long long kept = 0;
  for (long long t = 0; t < n; ++t) kept += get16(sb + 2 * t) != 0;
  const int sparse = kept * (r + 2) + (n + 7) / 8 < n * (r + 2);
  long long pos = pool_fill(L, cache, bh, n_cached), over = 0;
  for (long long t = 0; t < n; ++t) {
    const long long slot = n_cached + t, T = slot / 64;
    const int i = (int)(slot % 64);
    uint8_t* e = dir_entry(L, cache, bh, T);
    if (i == 0 || t == 0) { /* entering tile T */
      if (i == 0) {
        put32(e, (uint32_t)pos);
        put32(e + 4, 0);
        put64(e + 8, 0);
      } else { /* the chunk starts inside tile T: keep the rows below it */
        put64(e + 8, get64(e + 8) & (((uint64_t)1 << i) - 1));
      }
    }
    if (sparse && get16(sb + 2 * t) == 0) continue;
    if (pos >= L->pool) { ++over; continue; }
    memcpy(cache + L->k_coef + (bh * L->pool + pos) * r, codes + t * r, (size_t)r);
    put16(cache + L->k_cscale + (bh * L->pool + pos) * 2, get16(sb + 2 * t));
    put64(e + 8, get64(e + 8) | ((uint64_t)1 << i));
    ++pos;
  }
  uint8_t* oc = cache + L->k_over + bh * 4;
  put32(oc, get32(oc) + (uint32_t)over);
}

/* ----------------------------------------------------- INT2 residual (O3) */

static float clampf(float x, float lo, float hi) { return x < lo ? lo : (x > hi ? hi : x); }

/* Eq. 2 step size of one group: the residual range extended to contain 0, over
 * the 2^2 - 1 = 3 steps of q_min = 0 .. q_max = 3 (fp32). */
static float group_step(const float* x, const float* mu, int n, float* lo_out) {
  float lo = 0.0f, hi = 0.0f;
  for (int c = 0; c < n; ++c) {
    float r = x[c] - mu[c];
    if (r < lo) lo = r;
    if (r > hi) hi = r;
  }
  *lo_out = lo;
  return (hi - lo) / 3.0f;
}

void ora_int2_quantise(const float* x, const float* mu, int n, float step, uint8_t* codes,
                       uint8_t* zero_point, float* xhat) {
  /* Eq. 3 residual; Eq. 1-2 with the stored step; Eq. 4 reconstruction */
  float lo = 0.0f;
  (void)group_step(x, mu, n, &lo);
  int z = 0;
  if (step != 0.0f) z = (int)clampf(rintf(0.0f - lo / step), 0.0f, 3.0f);
  *zero_point = (uint8_t)z;
  for (int c = 0; c < n; ++c) {
    float r = x[c] - mu[c];
    int q = 0;
    if (step != 0.0f) q = (int)clampf(rintf(r / step) + (float)z, 0.0f, 3.0f); /* Eq. 1 */
    codes[c] = (uint8_t)q;
    xhat[c] = mu[c] + step * (float)(q - z); /* Eq. 4: centroid + dequantised residual */
  }
}

void ora_int2_group(const float* x, const float* mu, int n, uint8_t* codes,
                    uint8_t* zero_point, uint16_t* scale_f16, float* xhat) {
  /* the step size stored as FP16 (saturating), then the quantiser with it */
  float lo;
  float s = group_step(x, mu, n, &lo);
  if (s > 65504.0f) s = 65504.0f;
  double sh = ora_round_f16((double)s);
  *scale_f16 = ora_f16_bits(sh);
  ora_int2_quantise(x, mu, n, (float)sh, codes, zero_point, xhat);
}

void ora_scales_i8(const float* t, int ng, uint16_t* sigma_f16, uint8_t* codes, float* step_out) {
  /* App. D.1: 8-bit codes with one FP16 secondary scale; the largest step sets
   * the secondary scale, sigma = FP16(max_g t_g / 255), and c_g = RN(t_g / sigma) */
  float mx = 0.0f;
  for (int g = 0; g < ng; ++g)
    if (t[g] > mx) mx = t[g];
  float sg = mx / 255.0f;
  if (sg > 65504.0f) sg = 65504.0f;
  double sh = ora_round_f16((double)sg);
  *sigma_f16 = ora_f16_bits(sh);
  float sf = (float)sh;
  for (int g = 0; g < ng; ++g) {
    int c = sf != 0.0f ? (int)clampf(rintf(t[g] / sf), 0.0f, 255.0f) : 0;
    codes[g] = (uint8_t)c;
    step_out[g] = sf * (float)c; /* exact: 11-bit times 8-bit significands */
  }
}

void ora_coef_row(const float* C, int r, int8_t* codes, uint16_t* scale_f16) {
  /* App. D.1: one INT8 PSAC row with one FP16 scale, symmetric over +-127:
   * s = FP16(max_k |C_k| / 127) (saturating), code_k = RN(C_k / s) clamped to
   * [-127, 127], and all codes 0 when s is 0 */
  float amax = 0.0f;
  for (int k = 0; k < r; ++k)
    if (fabsf(C[k]) > amax) amax = fabsf(C[k]);
  float s = amax / 127.0f;
  if (s > 65504.0f) s = 65504.0f;
  double sh = ora_round_f16((double)s);
  float shf = (float)sh;
  for (int k = 0; k < r; ++k)
    codes[k] = (int8_t)(shf != 0.0f ? (int)clampf(rintf(C[k] / shf), -127.0f, 127.0f) : 0);
  *scale_f16 = ora_f16_bits(sh);
}

int ora_keep_row(const float* C, const int8_t* codes, float scale, const float* lam, int r) {
  float before = 0.0f, after = 0.0f;
  for (int k = 0; k < r; ++k) {
    float e = C[k] - (float)codes[k] * scale;
    before = before + lam[k] * (C[k] * C[k]);
    after = after + lam[k] * (e * e);
  }
  return after < before;
}

/* ------------------------------------------------------------ QSAC (O2) */

/* Eq. 9: Query-aware distance, fp32, channels in order. */
static float dq_distance(const float* k, const float* mu_j, const float* w, int d) {
  float acc = 0.0f;
  for (int c = 0; c < d; ++c) {
    float t = k[c] - mu_j[c];
    acc = acc + w[c] * (t * t);
  }
  return acc;
}

/* Eq. 10 and Eq. 12: sum over groups of W_g * R_g^2 with W_g = sum_{c in g} w_c. */
static float qsac_score(const float* k, const float* mu_j, const float* Wg, int d, int G) {
  float S = 0.0f;
  for (int g = 0; g < d / G; ++g) {
    float mx = -INFINITY, mn = INFINITY;
    for (int c = g * G; c < (g + 1) * G; ++c) {
      float r = k[c] - mu_j[c];
      if (r > mx) mx = r;
      if (r < mn) mn = r;
    }
    float R = mx - mn;
    S = S + Wg[g] * (R * R);
  }
  return S;
}

static void group_weights(const float* w, int d, int G, float* Wg) {
  for (int g = 0; g < d / G; ++g) {
    float s = 0.0f;
    for (int c = g * G; c < (g + 1) * G; ++c) s = s + w[c];
    Wg[g] = s;
  }
}

static int less_pair(float a, int ia, float b, int ib) { return a < b || (a == b && ia < ib); }

/* Top-M candidate set C_i by (distance, id), then the argmin of the Eq. 12
 * score over it (ties to the lower id). */
static int qsac_select(const float* k, const float* mu, const float* dist, const float* w, int n_centroids,
                       int d, int group_size, int top_m, int* cand) {
  float Wg[256];
  int taken[256] = {0};
  int M = top_m < n_centroids ? top_m : n_centroids;
  for (int m = 0; m < M; ++m) {
    int best = -1;
    for (int j = 0; j < n_centroids; ++j)
      if (!taken[j] && (best < 0 || less_pair(dist[j], j, dist[best], best))) best = j;
    taken[best] = 1;
    cand[m] = best;
  }
  group_weights(w, d, group_size, Wg);
  int z = -1;
  float Sz = 0.0f;
  for (int m = 0; m < M; ++m) {
    int j = cand[m];
    float S = qsac_score(k, mu + (long long)j * d, Wg, d, group_size);
    if (z < 0 || less_pair(S, j, Sz, z)) { z = j; Sz = S; }
  }
  return z;
}

int ora_qsac_assign(const float* k, const float* mu, const float* w, int n_centroids,
                    int d, int group_size, int top_m, int* cand) {
  float dist[256];
  for (int j = 0; j < n_centroids; ++j) dist[j] = dq_distance(k, mu + (long long)j * d, w, d);
  return qsac_select(k, mu, dist, w, n_centroids, d, group_size, top_m, cand);
}

/* The full quadratic form (k - mu_j)^T m (k - mu_j) of the diagonal-approximation
 * ablation (App. C), fp32: the matrix-vector product first, rows in order. */
static float full_distance(const float* k, const float* mu_j, const float* m, int d) {
  float e[256];
  for (int c = 0; c < d; ++c) e[c] = k[c] - mu_j[c];
  float acc = 0.0f;
  for (int c = 0; c < d; ++c) {
    float t = 0.0f;
    for (int c2 = 0; c2 < d; ++c2) t = t + m[(long long)c * d + c2] * e[c2];
    acc = acc + e[c] * t;
  }
  return acc;
}

int ora_qsac_assign_full(const float* k, const float* mu, const float* m, const float* w, int n_centroids,
                         int d, int group_size, int top_m, int* cand) {
  float dist[256];
  for (int j = 0; j < n_centroids; ++j) dist[j] = full_distance(k, mu + (long long)j * d, m, d);
  return qsac_select(k, mu, dist, w, n_centroids, d, group_size, top_m, cand);
}

int ora_nearest(const float* x, const float* mu, int n_centroids, int d) {
  int best = 0;
  float bd = 0.0f;
  for (int j = 0; j < n_centroids; ++j) {
    float acc = 0.0f;
    for (int c = 0; c < d; ++c) {
      float t = x[c] - mu[(long long)j * d + c];
      acc = acc + t * t;
    }
    if (j == 0 || acc < bd) { best = j; bd = acc; }
  }
  return best;
}

/* ----------------------------------------------------------- calibration */

int ora_eigh(const double* a_in, int n, double* lam, double* vecs_t) {
  double* a = (double*)malloc(sizeof(double) * n * n);
  double* v = (double*)malloc(sizeof(double) * n * n);
  int* order = (int*)malloc(sizeof(int) * n);
  if (!a || !v || !order) { free(a); free(v); free(order); return -2; }
  memcpy(a, a_in, sizeof(double) * n * n);
  for (int i = 0; i < n * n; ++i) v[i] = 0.0;
  for (int i = 0; i < n; ++i) v[i * n + i] = 1.0;
  double fro = 0.0;
  for (int i = 0; i < n * n; ++i) fro += a[i] * a[i];
  fro = sqrt(fro);
  /* Cyclic Jacobi: rotate each off-diagonal pair to zero until the off-diagonal
   * mass is negligible (Golub & Van Loan, Sec. 8.5). */
  for (int sweep = 0; sweep < 100; ++sweep) {
    double off = 0.0;
    for (int p = 0; p < n; ++p)
      for (int q = p + 1; q < n; ++q) off += a[p * n + q] * a[p * n + q];
    if (sqrt(off) <= 1e-15 * fro || off == 0.0) break;
    for (int p = 0; p < n - 1; ++p) {
      for (int q = p + 1; q < n; ++q) {
        double apq = a[p * n + q];
        if (apq == 0.0) continue;
        double theta = (a[q * n + q] - a[p * n + p]) / (2.0 * apq);
        double t = (theta >= 0 ? 1.0 : -1.0) / (fabs(theta) + sqrt(theta * theta + 1.0));
        double c = 1.0 / sqrt(t * t + 1.0), s = t * c;
        for (int k = 0; k < n; ++k) { /* A <- A J (columns p, q) */
          double akp = a[k * n + p], akq = a[k * n + q];
          a[k * n + p] = c * akp - s * akq;
          a[k * n + q] = s * akp + c * akq;
        }
        for (int k = 0; k < n; ++k) { /* A <- J^T A (rows p, q) */
          double apk = a[p * n + k], aqk = a[q * n + k];
          a[p * n + k] = c * apk - s * aqk;
          a[q * n + k] = s * apk + c * aqk;
        }
        for (int k = 0; k < n; ++k) { /* V <- V J */
          double vkp = v[k * n + p], vkq = v[k * n + q];
          v[k * n + p] = c * vkp - s * vkq;
          v[k * n + q] = s * vkp + c * vkq;
        }
      }
    }
  }
  /* Eq. 15 orders lambda_1 >= ... >= lambda_d; equal values keep their index. */
  for (int i = 0; i < n; ++i) order[i] = i;
  for (int i = 1; i < n; ++i) {
    int o = order[i], j = i - 1;
    while (j >= 0 && a[order[j] * n + order[j]] < a[o * n + o]) { order[j + 1] = order[j]; --j; }
    order[j + 1] = o;
  }
  for (int i = 0; i < n; ++i) {
    int o = order[i];
    lam[i] = a[o * n + o];
    int arg = 0;
    for (int k = 1; k < n; ++k)
      if (fabs(v[k * n + o]) > fabs(v[arg * n + o])) arg = k;
    double sg = v[arg * n + o] < 0 ? -1.0 : 1.0;
    for (int k = 0; k < n; ++k) vecs_t[(long long)i * n + k] = sg * v[k * n + o];
  }
  free(a); free(v); free(order);
  return 0;
}

static void kmeans(const ora_cfg* c, const float* x, long long xs, long long n, int iters,
                   float* mu /* [Kc][d] */) {
  int d = c->head_dim, K = c->n_centroids;
  int* assign = (int*)malloc(sizeof(int) * (n > 0 ? n : 1));
  double* sum = (double*)malloc(sizeof(double) * K * d);
  long long* cnt = (long long*)malloc(sizeof(long long) * K);
  float* row = (float*)malloc(sizeof(float) * d);
  for (int j = 0; j < K; ++j) {
    long long t = n > 0 ? ((long long)j * n) / K : 0;
    for (int ch = 0; ch < d; ++ch) mu[(long long)j * d + ch] = n > 0 ? (float)round_table(c, x[t * xs + ch]) : 0.0f;
  }
  for (int it = 0; it < iters && n > 0; ++it) {
    for (long long t = 0; t < n; ++t) {
      for (int ch = 0; ch < d; ++ch) row[ch] = x[t * xs + ch];
      assign[t] = ora_nearest(row, mu, K, d);
    }
    memset(sum, 0, sizeof(double) * K * d);
    memset(cnt, 0, sizeof(long long) * K);
    for (long long t = 0; t < n; ++t) {
      int j = assign[t];
      cnt[j] += 1;
      for (int ch = 0; ch < d; ++ch) sum[(long long)j * d + ch] += (double)x[t * xs + ch];
    }
    for (int j = 0; j < K; ++j)
      if (cnt[j] > 0)
        for (int ch = 0; ch < d; ++ch)
          mu[(long long)j * d + ch] = (float)round_table(c, sum[(long long)j * d + ch] / (double)cnt[j]);
  }
  free(assign); free(sum); free(cnt); free(row);
}

int ora_calibrate(const ora_cfg* cfg, const float* q_hist, long long n_hist,
                  const float* k_cal, const float* v_cal, long long n_cal, int kmeans_iters,
                  float* mu_k, float* mu_v, float* w, float* u_t, float* lam, float* m_out) {
  if (!valid_cfg(cfg) || n_hist < 0 || n_cal < 0 || kmeans_iters < 0) return -1;
  if ((n_hist > 0 && !q_hist) || (n_cal > 0 && (!k_cal || !v_cal))) return -1;
  if (!mu_k || !mu_v || !w || (cfg->rank > 0 && (!u_t || !lam))) return -1;
  const int d = cfg->head_dim, H = cfg->heads, K = cfg->n_centroids, r = cfg->rank;
  const int nbh = cfg->batch * H;
  int err = 0;
#pragma omp parallel for schedule(dynamic)
  for (int bh = 0; bh < nbh; ++bh) {
    int b = bh / H, h = bh % H;
    long long tok_stride = (long long)H * d;
    float* wo = w + (long long)bh * d;
    float* uo = u_t + (long long)bh * r * d;
    float* lo = lam + (long long)bh * r;
    /* Eq. 6: historical Query second moment, fp64, tokens in order. */
    double* M = (double*)calloc((size_t)d * d, sizeof(double));
    double* lam_all = (double*)malloc(sizeof(double) * d);
    double* vec_t = (double*)malloc(sizeof(double) * d * d);
    if (!M || !lam_all || !vec_t) { err = -2; free(M); free(lam_all); free(vec_t); continue; }
    const float* qb = q_hist + (long long)b * n_hist * tok_stride + (long long)h * d;
    for (long long t = 0; t < n_hist; ++t) {
      const float* q = qb + t * tok_stride;
      for (int i = 0; i < d; ++i)
        for (int j = 0; j < d; ++j) M[i * d + j] += (double)q[i] * (double)q[j];
    }
    double tr = 0.0;
    if (n_hist > 0) {
      for (int i = 0; i < d * d; ++i) M[i] /= (double)n_hist;
      for (int i = 0; i < d; ++i) tr += M[i * d + i];
    }
    float* mo = m_out ? m_out + (long long)bh * d * d : NULL;
    if (n_hist == 0 || tr == 0.0) {
      /* cold start: uniform sensitivity, PSAC inactive */
      for (int c = 0; c < d; ++c) wo[c] = 1.0f;
      for (long long i = 0; i < (long long)r * d; ++i) uo[i] = 0.0f;
      for (int k = 0; k < r; ++k) lo[k] = 0.0f;
      if (mo)
        for (int i = 0; i < d * d; ++i) mo[i] = (i / d == i % d) ? 1.0f : 0.0f;
    } else {
      /* the full metric: M over the mean of its diagonal, so its diagonal is w */
      if (mo)
        for (int i = 0; i < d * d; ++i) mo[i] = (float)(M[i] / (tr / (double)d));
      /* Eq. 8: w_c = M_cc / ((1/d) sum_c' M_c'c') */
      for (int c = 0; c < d; ++c) wo[c] = (float)(M[c * d + c] / (tr / (double)d));
      /* Eq. 15-16: top-r eigenvectors of M */
      ora_eigh(M, d, lam_all, vec_t);
      for (int k = 0; k < r; ++k) {
        lo[k] = (float)lam_all[k];
        for (int c = 0; c < d; ++c) uo[(long long)k * d + c] = (float)round_table(cfg, vec_t[(long long)k * d + c]);
      }
    }
    free(M); free(lam_all); free(vec_t);
    /* Eq. 3: centroids by K-means on the calibration tokens, Keys and Values apart. */
    kmeans(cfg, k_cal + (long long)b * n_cal * tok_stride + (long long)h * d, tok_stride, n_cal,
           kmeans_iters, mu_k + (long long)bh * K * d);
    kmeans(cfg, v_cal + (long long)b * n_cal * tok_stride + (long long)h * d, tok_stride, n_cal,
           kmeans_iters, mu_v + (long long)bh * K * d);
  }
  return err;
}

/* ------------------------------------------------------------- append */

static void put_codes(uint8_t* dst, const uint8_t* q, int d) {
  for (int i = 0; i < d / 4; ++i)
    dst[i] = (uint8_t)(q[4 * i] | (q[4 * i + 1] << 2) | (q[4 * i + 2] << 4) | (q[4 * i + 3] << 6));
}

/* One token: centroid + per-group INT2 residual, written at slot pointers. With
 * SCALE_I8 all group steps are found first: they share the secondary scale. */
static void store_residual(const layout* L, int G, const float* x, const float* mu_z,
                           uint8_t* codes_dst, uint8_t* zp_dst, uint8_t* scale_dst, uint8_t* sigma_dst,
                           float* xhat) {
  uint8_t q[256];
  memset(zp_dst, 0, (size_t)L->zpb);
  if (L->i8) {
    float t[256], step[256], lo;
    uint16_t sigma;
    for (int g = 0; g < L->ng; ++g) t[g] = group_step(x + g * G, mu_z + g * G, G, &lo);
    ora_scales_i8(t, L->ng, &sigma, scale_dst, step);
    put16(sigma_dst, sigma);
    for (int g = 0; g < L->ng; ++g) {
      uint8_t zg;
      ora_int2_quantise(x + g * G, mu_z + g * G, G, step[g], q + g * G, &zg, xhat + g * G);
      zp_dst[g / 4] |= (uint8_t)(zg << (2 * (g % 4)));
    }
  } else {
    for (int g = 0; g < L->ng; ++g) {
      uint8_t zg;
      uint16_t sg;
      ora_int2_group(x + g * G, mu_z + g * G, G, q + g * G, &zg, &sg, xhat + g * G);
      zp_dst[g / 4] |= (uint8_t)(zg << (2 * (g % 4)));
      put16(scale_dst + 2 * g, sg);
    }
  }
  put_codes(codes_dst, q, L->d);
}

int ora_append(const ora_cfg* cfg, const float* mu_k, const float* mu_v, const float* w,
               const float* u_t, const float* lam, const float* m_full, uint8_t* cache, long long n_cached,
               const float* k_new, const float* v_new, long long n_new,
               float* coef_f32, int* k_ids, int* v_ids, int* cand) {
  if (!valid_cfg(cfg) || n_cached < 0 || n_new < 0) return -1;
  if (n_cached + n_new > cfg->capacity) return -3;
  if ((cfg->storage & ORA_STORE_SPARSE) && n_new > cfg->coef_stage) return -3;
  if (n_new == 0) return 0;
  if (!mu_k || !mu_v || !w || !cache || !k_new || !v_new || (cfg->rank > 0 && !u_t)) return -1;
  const int gate = (cfg->storage & ORA_STORE_GATE) && cfg->rank > 0;
  if (gate && !lam) return -1;
  const int full = cfg->metric == ORA_METRIC_FULL;
  if (full && !m_full) return -1;
  const layout L = make_layout(cfg);
  const int d = cfg->head_dim, H = cfg->heads, K = cfg->n_centroids, r = cfg->rank, G = cfg->group_size;
  const int M = cfg->top_m < K ? cfg->top_m : K;
  const int nbh = cfg->batch * H;
#pragma omp parallel for schedule(dynamic)
  for (int bh = 0; bh < nbh; ++bh) {
    int b = bh / H, h = bh % H;
    const float* muk = mu_k + (long long)bh * K * d;
    const float* muv = mu_v + (long long)bh * K * d;
    const float* wh = w + (long long)bh * d;
    const float* uh = u_t + (long long)bh * r * d;
    float xhat[256];
    int cands[256];
    /* SPARSE: the chunk's rows go to the staging rows, then sparse_commit */
    int8_t* st_codes = L.sparse ? (int8_t*)(cache + L.k_st_codes + (long long)bh * L.stage * r) : NULL;
    uint8_t* st_scale = L.sparse ? cache + L.k_st_scale + (long long)bh * L.stage * 2 : NULL;
    for (long long t = 0; t < n_new; ++t) {
      long long slot = (long long)bh * L.slots + n_cached + t;
      long long src = (((long long)b * n_new + t) * H + h) * d;
      const float* k = k_new + src;
      const float* v = v_new + src;
      long long diag = ((long long)bh * n_new + t);
      /* QSAC: top-M by Eq. 9 (or the full form), then argmin of Eq. 12 */
      int z = full ? ora_qsac_assign_full(k, muk, m_full + (long long)bh * d * d, wh, K, d, G, M, cands)
                   : ora_qsac_assign(k, muk, wh, K, d, G, M, cands);
      cache[L.k_ids + slot] = (uint8_t)z;
      store_residual(&L, G, k, muk + (long long)z * d, cache + L.k_codes + slot * (d / 4),
                     cache + L.k_zp + slot * L.zpb, cache + L.k_scale + slot * L.sb, cache + L.k_sigma + slot * 2,
                     xhat);
      if (k_ids) k_ids[diag] = z;
      if (cand) for (int m = 0; m < M; ++m) cand[diag * M + m] = cands[m];
      if (r > 0) {
        /* Eq. 13 and Eq. 16: C = (k - khat_0) U_r, fp64 */
        float Cf[256];
        for (int kk = 0; kk < r; ++kk) {
          double acc = 0.0;
          for (int c = 0; c < d; ++c) acc += ((double)k[c] - (double)xhat[c]) * (double)uh[(long long)kk * d + c];
          Cf[kk] = (float)acc;
          if (coef_f32) coef_f32[diag * r + kk] = Cf[kk];
        }
        /* INT8 row with one FP16 scale (App. D.1) */
        int8_t* code = L.sparse ? st_codes + t * r : (int8_t*)(cache + L.k_coef + slot * r);
        uint16_t sbits;
        ora_coef_row(Cf, r, code, &sbits);
        /* App. D.1 retention: a row that does not lower the error is zeroed */
        if (gate && !ora_keep_row(Cf, code, (float)ora_f16_value(sbits), lam + (long long)bh * r, r)) {
          memset(code, 0, (size_t)r);
          sbits = 0;
        }
        put16(L.sparse ? st_scale + 2 * t : cache + L.k_cscale + slot * 2, sbits);
      }
      /* Values: nearest centroid, same residual path, no PSAC */
      int zv = ora_nearest(v, muv, K, d);
      cache[L.v_ids + slot] = (uint8_t)zv;
      store_residual(&L, G, v, muv + (long long)zv * d, cache + L.v_codes + slot * (d / 4),
                     cache + L.v_zp + slot * L.zpb, cache + L.v_scale + slot * L.sb, cache + L.v_sigma + slot * 2,
                     xhat);
      if (v_ids) v_ids[diag] = zv;
    }
    if (L.sparse) sparse_commit(&L, cache, bh, n_cached, n_new);
  }
  return 0;
}

/* ------------------------------------------------------------- decode */

static void load_residual(const layout* L, int G, const uint8_t* codes, const uint8_t* zp,
                          const uint8_t* scale, const uint8_t* sigma, const float* mu_z, double* out) {
  for (int c = 0; c < L->d; ++c) {
    int g = c / G;
    int q = (codes[c / 4] >> (2 * (c % 4))) & 3;
    int z = (zp[g / 4] >> (2 * (g % 4))) & 3;
    float s = L->i8 ? (float)ora_f16_value(get16(sigma)) * (float)scale[g]
                    : (float)ora_f16_value(get16(scale + 2 * g));
    out[c] = (double)(mu_z[c] + s * (float)(q - z)); /* Eq. 4, fp32 as when encoding */
  }
}

/* ------------------------------------------- per-chunk coefficient layout */


/* the chunk records read slot-addressed rows: not a SPARSE cache */
static int coef_args_ok(const ora_cfg* cfg, long long start, long long n) {
  return valid_cfg(cfg) && cfg->rank > 0 && !(cfg->storage & ORA_STORE_SPARSE) && start >= 0 && n >= 0 &&
         n <= 65536 && start + n <= cfg->capacity;
}

/* kept rows (non-zero FP16 scale) of head bh in the chunk */
static long long coef_kept(const layout* L, const uint8_t* cache, long long bh, long long start, long long n) {
  long long k = 0;
  for (long long t = start; t < start + n; ++t) k += get16(cache + L->k_cscale + (bh * L->slots + t) * 2) != 0;
  return k;
}

long long ora_coef_record_bytes(const ora_cfg* cfg, const uint8_t* cache, long long start, long long n, int* layout_out) {
  if (!coef_args_ok(cfg, start, n) || !cache) return -1;
  const layout L = make_layout(cfg);
  const long long nbh = (long long)cfg->batch * cfg->heads, r = cfg->rank;
  long long kept = 0;
  for (long long bh = 0; bh < nbh; ++bh) kept += coef_kept(&L, cache, bh, start, n);
  const long long dense = 16 + nbh * n * (r + 2), sparse = 16 + 4 * nbh + kept * (r + 4);
  const int lay = sparse < dense ? ORA_COEF_SPARSE : ORA_COEF_DENSE;
  if (layout_out) *layout_out = lay;
  return lay == ORA_COEF_SPARSE ? sparse : dense;
}

int ora_coef_pack(const ora_cfg* cfg, const uint8_t* cache, long long start, long long n, uint8_t* out,
                  long long out_bytes, long long* written) {
  int lay;
  const long long need = ora_coef_record_bytes(cfg, cache, start, n, &lay);
  if (need < 0 || !out) return -1;
  if (out_bytes < need) return -3;
  const layout L = make_layout(cfg);
  const long long nbh = (long long)cfg->batch * cfg->heads, r = cfg->rank;
  put32(out, (uint32_t)lay);
  put32(out + 4, (uint32_t)n);
  put32(out + 8, (uint32_t)r);
  put32(out + 12, (uint32_t)nbh);
  if (lay == ORA_COEF_DENSE) {
    uint8_t* codes = out + 16;
    uint8_t* scales = codes + nbh * n * r;
    for (long long bh = 0; bh < nbh; ++bh)
      for (long long t = 0; t < n; ++t) {
        const long long slot = bh * L.slots + start + t, row = bh * n + t;
        memcpy(codes + row * r, cache + L.k_coef + slot * r, (size_t)r);
        memcpy(scales + row * 2, cache + L.k_cscale + slot * 2, 2);
      }
  } else {
    uint8_t* p = out + 16 + 4 * nbh;
    for (long long bh = 0; bh < nbh; ++bh) {
      const long long cnt = coef_kept(&L, cache, bh, start, n);
      put32(out + 16 + 4 * bh, (uint32_t)cnt);
      uint8_t* idx = p;
      uint8_t* codes = idx + 2 * cnt;
      uint8_t* scales = codes + r * cnt;
      long long m = 0;
      for (long long t = 0; t < n; ++t) {
        const long long slot = bh * L.slots + start + t;
        if (get16(cache + L.k_cscale + slot * 2) == 0) continue;
        put16(idx + 2 * m, (uint16_t)t);
        memcpy(codes + m * r, cache + L.k_coef + slot * r, (size_t)r);
        memcpy(scales + 2 * m, cache + L.k_cscale + slot * 2, 2);
        ++m;
      }
      p = scales + 2 * cnt;
    }
  }
  if (written) *written = need;
  return 0;
}

int ora_coef_unpack(const ora_cfg* cfg, const uint8_t* rec, long long rec_bytes, uint8_t* cache, long long start,
                    long long n) {
  if (!coef_args_ok(cfg, start, n) || !rec || !cache || rec_bytes < 16) return -1;
  const layout L = make_layout(cfg);
  const long long nbh = (long long)cfg->batch * cfg->heads, r = cfg->rank;
  const uint32_t lay = get32(rec);
  if (get32(rec + 4) != (uint32_t)n || get32(rec + 8) != (uint32_t)r || get32(rec + 12) != (uint32_t)nbh) return -1;
  if (lay == ORA_COEF_DENSE) {
    if (rec_bytes < 16 + nbh * n * (r + 2)) return -1;
    const uint8_t* codes = rec + 16;
    const uint8_t* scales = codes + nbh * n * r;
    for (long long bh = 0; bh < nbh; ++bh)
      for (long long t = 0; t < n; ++t) {
        const long long slot = bh * L.slots + start + t, row = bh * n + t;
        memcpy(cache + L.k_coef + slot * r, codes + row * r, (size_t)r);
        memcpy(cache + L.k_cscale + slot * 2, scales + row * 2, 2);
      }
    return 0;
  }
  if (lay != ORA_COEF_SPARSE || rec_bytes < 16 + 4 * nbh) return -1;
  long long total = 16 + 4 * nbh;
  for (long long bh = 0; bh < nbh; ++bh) total += (long long)get32(rec + 16 + 4 * bh) * (r + 4);
  if (rec_bytes < total) return -1;
  const uint8_t* p = rec + 16 + 4 * nbh;
  for (long long bh = 0; bh < nbh; ++bh) {
    const long long cnt = get32(rec + 16 + 4 * bh);
    if (cnt > n) return -1;
    for (long long t = 0; t < n; ++t) {
      const long long slot = bh * L.slots + start + t;
      memset(cache + L.k_coef + slot * r, 0, (size_t)r);
      memset(cache + L.k_cscale + slot * 2, 0, 2);
    }
    const uint8_t* idx = p;
    const uint8_t* codes = idx + 2 * cnt;
    const uint8_t* scales = codes + r * cnt;
    for (long long m = 0; m < cnt; ++m) {
      const long long t = get16(idx + 2 * m);
      if (t >= n) return -1;
      const long long slot = bh * L.slots + start + t;
      memcpy(cache + L.k_coef + slot * r, codes + m * r, (size_t)r);
      memcpy(cache + L.k_cscale + slot * 2, scales + 2 * m, 2);
    }
    p = scales + 2 * cnt;
  }
  return 0;
}

int ora_decode(const ora_cfg* cfg, const float* mu_k, const float* mu_v,
               const uint8_t* cache, int b, int h, long long n,
               double* k0, double* chat, double* v) {
  if (!valid_cfg(cfg) || b < 0 || b >= cfg->batch || h < 0 || h >= cfg->heads || n < 0 || n > cfg->capacity)
    return -1;
  const layout L = make_layout(cfg);
  const int d = cfg->head_dim, K = cfg->n_centroids, r = cfg->rank, G = cfg->group_size;
  long long bh = (long long)b * cfg->heads + h;
  for (long long t = 0; t < n; ++t) {
    long long slot = bh * L.slots + t;
    int zk = cache[L.k_ids + slot], zv = cache[L.v_ids + slot];
    if (zk >= K || zv >= K) return -4;
    if (k0)
      load_residual(&L, G, cache + L.k_codes + slot * (d / 4), cache + L.k_zp + slot * L.zpb,
                    cache + L.k_scale + slot * L.sb, cache + L.k_sigma + slot * 2, mu_k + (bh * K + zk) * d,
                    k0 + t * d);
    if (v)
      load_residual(&L, G, cache + L.v_codes + slot * (d / 4), cache + L.v_zp + slot * L.zpb,
                    cache + L.v_scale + slot * L.sb, cache + L.v_sigma + slot * 2, mu_v + (bh * K + zv) * d,
                    v + t * d);
    if (chat && r > 0) {
      long long row = slot;
      if (L.sparse) {
        const long long pr = pool_row(&L, cache, bh, t);
        if (pr >= L.pool) return -5; /* a directory pointing past the pool */
        row = pr < 0 ? -1 : bh * L.pool + pr;
      }
      if (row < 0) {
        for (int kk = 0; kk < r; ++kk) chat[t * r + kk] = 0.0;
      } else {
        float s = (float)ora_f16_value(get16(cache + L.k_cscale + row * 2));
        const int8_t* code = (const int8_t*)(cache + L.k_coef + row * r);
        for (int kk = 0; kk < r; ++kk) chat[t * r + kk] = (double)((float)code[kk] * s);
      }
    }
  }
  return 0;
}

/* ------------------------------------------------------------- attend */

static int cmp_rows(const void* a, const void* b) {
  const int* x = (const int*)a;
  const int* y = (const int*)b;
  if (x[0] != y[0]) return x[0] - y[0];
  if (x[1] != y[1]) return x[1] - y[1];
  return x[2] - y[2];
}

int ora_attend(const ora_cfg* cfg, const float* mu_k, const float* mu_v, const float* u_t,
               const uint8_t* cache, long long n_cache, const float* q, long long n_q,
               long long q_start, int frame_tokens, const float* coef_override,
               int n_rows, const int* rows, double* out, double* lse, double* logits) {
  return ora_attend_active(cfg, mu_k, mu_v, u_t, cache, n_cache, NULL, NULL, 0, q, n_q, q_start, frame_tokens,
                           coef_override, n_rows, rows, out, lse, logits);
}

/* Keys [0, n_cache) are decoded from the packed cache; keys [n_cache, n_cache +
 * n_act) are the exact active-chunk tokens, rounded to the table type like every
 * other operand, with no PSAC term (only completed chunks are packed). */
int ora_attend_active(const ora_cfg* cfg, const float* mu_k, const float* mu_v, const float* u_t,
                      const uint8_t* cache, long long n_cache, const float* k_act, const float* v_act,
                      long long n_act, const float* q, long long n_q, long long q_start, int frame_tokens,
                      const float* coef_override, int n_rows, const int* rows, double* out, double* lse,
                      double* logits) {
  const long long start0 = 0;
  return ora_attend_epochs(cfg, 1, &start0, mu_k, mu_v, u_t, cache, n_cache, k_act, v_act, n_act, q, n_q, q_start,
                           frame_tokens, coef_override, n_rows, rows, out, lse, logits);
}

/* Keys [epoch_start[e], epoch_start[e+1]) of the packed cache were appended with
 * the tables of epoch e (centroids and U_r of that epoch, Sec. 5 streaming):
 * their Khat_0 and Vhat decode with epoch e's centroids, and their PSAC term is
 * (q U_r^(e)) . chat (Eq. 17 with the epoch's own subspace). Tables are
 * [n_epochs][B][H][...]; epoch_start[0] = 0 and increases. */
int ora_attend_epochs(const ora_cfg* cfg, int n_epochs, const long long* epoch_start, const float* mu_k,
                      const float* mu_v, const float* u_t, const uint8_t* cache, long long n_cache,
                      const float* k_act, const float* v_act, long long n_act, const float* q, long long n_q,
                      long long q_start, int frame_tokens, const float* coef_override, int n_rows, const int* rows,
                      double* out, double* lse, double* logits) {
  if (!valid_cfg(cfg) || n_cache < 0 || n_cache > cfg->capacity || n_act < 0 || (n_act > 0 && (!k_act || !v_act)) ||
      n_q < 0 || q_start < 0 || q_start > n_cache + n_act || frame_tokens < 1 || n_rows < 0 || n_epochs < 1 ||
      !epoch_start || epoch_start[0] != 0)
    return -1;
  for (int e = 1; e < n_epochs; ++e)
    if (epoch_start[e] <= epoch_start[e - 1]) return -1;
  const long long n_all = n_cache + n_act;
  const int d = cfg->head_dim, H = cfg->heads, r = cfg->rank;
  const long long tab_mu = (long long)cfg->batch * H * cfg->n_centroids * d;  /* floats per epoch */
  const long long tab_u = (long long)cfg->batch * H * (r > 0 ? r : 1) * d;
  /* rows sorted by head so that each head's cache is decoded once; idx[4] keeps
   * the caller's row number */
  int* srt = (int*)malloc(sizeof(int) * 4 * (n_rows > 0 ? n_rows : 1));
  for (int i = 0; i < n_rows; ++i) {
    srt[4 * i] = rows[3 * i]; srt[4 * i + 1] = rows[3 * i + 1]; srt[4 * i + 2] = rows[3 * i + 2];
    srt[4 * i + 3] = i;
    if (rows[3 * i] < 0 || rows[3 * i] >= cfg->batch || rows[3 * i + 1] < 0 || rows[3 * i + 1] >= H ||
        rows[3 * i + 2] < 0 || rows[3 * i + 2] >= n_q) { free(srt); return -1; }
  }
  qsort(srt, (size_t)n_rows, sizeof(int) * 4, cmp_rows);
  const long long nd = n_all > 0 ? n_all : 1, nc1 = n_cache > 0 ? n_cache : 1;
  double* K0 = (double*)malloc(sizeof(double) * nd * d);
  double* V = (double*)malloc(sizeof(double) * nd * d);
  double* Ch = (double*)malloc(sizeof(double) * nd * (r > 0 ? r : 1));
  double* tk = (double*)malloc(sizeof(double) * nc1 * d);
  double* tv = (double*)malloc(sizeof(double) * nc1 * d);
  double* tc = (double*)malloc(sizeof(double) * nc1 * (r > 0 ? r : 1));
  int* ep = (int*)malloc(sizeof(int) * nd);
  if (!K0 || !V || !Ch || !tk || !tv || !tc || !ep) {
    free(srt); free(K0); free(V); free(Ch); free(tk); free(tv); free(tc); free(ep);
    return -2;
  }
  for (long long j = 0, e = 0; j < n_all; ++j) {
    while (e + 1 < n_epochs && j >= epoch_start[e + 1]) ++e;
    ep[j] = (int)e;
  }
  const double inv_sqrt_d = 1.0 / sqrt((double)d);
  int i0 = 0, status = 0;
  while (i0 < n_rows) {
    int b = srt[4 * i0], h = srt[4 * i0 + 1], i1 = i0;
    while (i1 < n_rows && srt[4 * i1] == b && srt[4 * i1 + 1] == h) ++i1;
    long long bh = (long long)b * H + h;
    /* each epoch's keys decode with that epoch's centroids */
    for (int e = 0; e < n_epochs && status == 0; ++e) {
      const long long s0 = epoch_start[e], s1 = e + 1 < n_epochs ? epoch_start[e + 1] : n_cache;
      if (s0 >= n_cache) break;
      if (ora_decode(cfg, mu_k + e * tab_mu, mu_v + e * tab_mu, cache, b, h, n_cache, tk, tc, tv)) { status = -4; break; }
      for (long long j = s0; j < s1 && j < n_cache; ++j) {
        memcpy(K0 + j * d, tk + j * d, sizeof(double) * d);
        memcpy(V + j * d, tv + j * d, sizeof(double) * d);
        if (r > 0) memcpy(Ch + j * r, tc + j * r, sizeof(double) * r);
      }
    }
    if (status) break;
    /* operands of the attention product, in the table type (BF16 per App. D.1) */
    for (long long t = 0; t < n_cache * d; ++t) { K0[t] = round_table(cfg, K0[t]); V[t] = round_table(cfg, V[t]); }
    for (long long t = 0; t < n_cache * r; ++t)
      Ch[t] = coef_override ? (double)coef_override[bh * n_cache * r + t] : round_table(cfg, Ch[t]);
    for (long long j = 0; j < n_act; ++j) {
      const long long src = (((long long)b * n_act + j) * H + h) * d;
      for (int c = 0; c < d; ++c) {
        K0[(n_cache + j) * d + c] = round_table(cfg, (double)k_act[src + c]);
        V[(n_cache + j) * d + c] = round_table(cfg, (double)v_act[src + c]);
      }
      for (int kk = 0; kk < r; ++kk) Ch[(n_cache + j) * r + kk] = 0.0;
    }
#pragma omp parallel for schedule(dynamic)
    for (int ri = i0; ri < i1; ++ri) {
      long long i = srt[4 * ri + 2];
      int dst = srt[4 * ri + 3];
      const float* qi = q + (((long long)b * n_q + i) * H + h) * d;
      /* q U_r^(e) of every epoch, in the table type */
      double* u = (double*)malloc(sizeof(double) * n_epochs * (r > 0 ? r : 1));
      for (int e = 0; e < n_epochs; ++e)
        for (int kk = 0; kk < r; ++kk) {
          double acc = 0.0;
          const float* ur = u_t + e * tab_u + (bh * r + kk) * d;
          for (int c = 0; c < d; ++c) acc += (double)qi[c] * (double)ur[c];
          u[e * r + kk] = round_table(cfg, acc);
        }
      double* L = (double*)malloc(sizeof(double) * nd);
      double m = -INFINITY;
      for (long long j = 0; j < n_all; ++j) {
        int visible = j < q_start || (j - q_start) / frame_tokens <= i / frame_tokens;
        if (!visible) { L[j] = -INFINITY; continue; }
        /* Eq. 5 with Eq. 17: (q khat_0 + (q U_r) c) / sqrt(d), U_r of the key's epoch */
        double acc = 0.0;
        for (int c = 0; c < d; ++c) acc += (double)qi[c] * K0[j * d + c];
        for (int kk = 0; kk < r; ++kk) acc += u[ep[j] * r + kk] * Ch[j * r + kk];
        L[j] = acc * inv_sqrt_d;
        if (L[j] > m) m = L[j];
      }
      double l = 0.0;
      double* o = out + (long long)dst * d;
      for (int c = 0; c < d; ++c) o[c] = 0.0;
      if (m > -INFINITY) {
        for (long long j = 0; j < n_all; ++j) {
          if (L[j] == -INFINITY) continue;
          double p = exp(L[j] - m);
          l += p;
          for (int c = 0; c < d; ++c) o[c] += p * V[j * d + c];
        }
        for (int c = 0; c < d; ++c) o[c] /= l;
        lse[dst] = m + log(l);
      } else {
        lse[dst] = -INFINITY;
      }
      if (logits) memcpy(logits + (long long)dst * n_all, L, sizeof(double) * n_all);
      free(L);
      free(u);
    }
    i0 = i1;
  }
  free(srt); free(K0); free(V); free(Ch); free(tk); free(tv); free(tc); free(ep);
  return status;
}

int ora_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void ora_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
