/*
 * QuantWM CPU oracle: TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-unit-at-a-time CPU implementation of what the QuantWM
 * hot path computes, written from the paper (arxiv 2609.26425, Sections 2, 4.1,
 * 4.2 and Appendix D.1). Only tests/, the package's smoke check and the
 * benchmark's CPU-baseline leg may load it. It shares no code with the HIP
 * library; the two only agree on the packed byte format of the cache.
 *
 * Precision. Attention, second moments, eigendecomposition and PSAC
 * coefficients are computed in fp64. Every decision that turns a float into an
 * integer (the Eq. 9 distance, the Eq. 12 score, the INT2 quantiser of Eq. 1-2,
 * the INT8 coefficient codes, the K-means assignment) is taken in fp32, the
 * precision of the GPU kernels, evaluated in the order the equations are written
 * (IEEE division, round-to-nearest-even, no contraction).
 *
 * Layouts. Activations are float32 arrays [B, N, H, d] (token-major) holding
 * values that are exact in the workload's element type. Method-level tables are
 * float32 arrays: centroids [B, H, Kc, d], sensitivities w [B, H, d], principal
 * basis U_r^T [B, H, r, d] (row k = k-th eigenvector), eigenvalues [B, H, r].
 *
 * Every function returns 0 on success and a negative number on a bad argument.
 */
#ifndef QUANTWM_ORACLE_H
#define QUANTWM_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int batch, heads, head_dim;  /* B, H, d (d <= 256, a multiple of 4) */
  int n_centroids;             /* Kc <= 256 (uint8 centroid ids, App. D.1) */
  int group_size;              /* G: INT2 residual group along channels */
  int rank;                    /* r: PSAC rank (0 disables PSAC) */
  int top_m;                   /* M: QSAC candidate count (Sec. 4.1) */
  long long capacity;          /* cache slots per (b, h) */
  int table_bf16;              /* 1: centroids, U_r and attention operands are BF16 */
  int storage;                 /* ORA_STORE_* flags (App. D.1 packed-storage options) */
  int metric;                  /* ORA_METRIC_*: the distance of the QSAC candidate search */
  long long coef_rows;         /* ORA_STORE_SPARSE: PSAC rows the pool of each (b, h) holds (0 = slots) */
  long long coef_stage;        /* ORA_STORE_SPARSE: largest chunk (tokens) one append call takes */
} ora_cfg;

/* App. D.1 storage options. SCALE_I8: the group step sizes of a token-head are
 * stored as 8-bit codes c_g in [0, 255] with one FP16 secondary scale sigma shared
 * by the token-head's groups; the step is sigma * c_g. GATE: a PSAC row is kept
 * only when it lowers the Query-weighted error approximated on the principal
 * subspace (sum_k lam_k C_k^2 before, sum_k lam_k (C_k - chat_k)^2 after);
 * otherwise its codes and scale are zero. */
#define ORA_STORE_SCALE_I8 1
#define ORA_STORE_GATE 2
/* SPARSE (needs rank >= 1): the PSAC rows live in a row pool per (b, h) with a
 * directory per 64-slot tile, {u32 base, u32 0, u64 mask}: bit i of the mask
 * says that slot 64 T + i has a row in the pool, at row base + (set bits below
 * i). Rows are stored in slot order. Each append call (one chunk) stores, per
 * (b, h), either every row of the chunk (dense) or only its rows with a
 * non-zero scale (sparse), whichever is smaller counting one mask bit per slot
 * as the sparse index: sparse iff kept (r + 2) + ceil(n / 8) < n (r + 2).
 * A row past the pool's end is not stored (bit clear: no correction) and
 * counted in the per-(b, h) u32 overflow counter. A slot without a row reads
 * as a zero PSAC row. Sections: K coef and K cscale hold [B*H][coef_rows] rows;
 * then, after the secondary scales, the directory [B*H][slots/64][16 B], the
 * overflow counters [B*H] u32, and the staging rows of one append call,
 * codes [B*H][coef_stage][r] and scales [B*H][coef_stage] (the chunk's rows
 * are written there first; an append of more than coef_stage tokens is
 * refused). */
#define ORA_STORE_SPARSE 4

/* QSAC candidate metric. DIAG: Eq. 9, the channel-weighted distance with w, the
 * diagonal of the normalised Query second moment. FULL: the full quadratic form
 * of App. C (the diagonal-approximation ablation), (k - mu)^T Mn (k - mu) with
 * Mn = M / ((1/d) tr M), whose diagonal is w; the ranking is the same for any
 * positive multiple of M. At cold start Mn is the identity. The candidate score
 * (Eq. 10-12) and everything after it are unchanged. */
#define ORA_METRIC_DIAG 0
#define ORA_METRIC_FULL 1

/* Packed cache size in bytes and the per-token-head byte counts (K and V). */
long long ora_cache_bytes(const ora_cfg* cfg);
int ora_token_bytes(const ora_cfg* cfg, int* k_bytes, int* v_bytes);

/* Number conversions the format fixes (round to nearest, ties to even). */
double ora_round_bf16(double x);
double ora_round_f16(double x);  /* IEEE binary16, subnormals kept, overflow -> inf */
uint16_t ora_f16_bits(double exact_f16_value);
double ora_f16_value(uint16_t bits);

/* Eq. 1-2 with b = 2 on one residual group, plus Eq. 4 reconstruction. */
void ora_int2_group(const float* x, const float* mu, int n, uint8_t* codes,
                    uint8_t* zero_point, uint16_t* scale_f16, float* xhat);

/* The same with the step size given (the stored scale): Eq. 1-2 codes and
 * zero-point for the group's residual range, Eq. 4 reconstruction. */
void ora_int2_quantise(const float* x, const float* mu, int n, float step, uint8_t* codes,
                       uint8_t* zero_point, float* xhat);

/* SCALE_I8: the fp32 step sizes t[0..ng) of one token-head -> FP16 secondary
 * scale (bits) and 8-bit codes; step_out[g] = sigma * c_g. */
void ora_scales_i8(const float* t, int ng, uint16_t* sigma_f16, uint8_t* codes, float* step_out);

/* App. D.1 INT8 PSAC row of r coefficients C: FP16 scale s = RN16(max|C|/127)
 * (bits to *scale_f16), codes RN(C/s) clamped to [-127, 127], 0 when s is 0. */
void ora_coef_row(const float* C, int r, int8_t* codes, uint16_t* scale_f16);

/* GATE: 1 when the INT8 row chat (codes * scale) lowers the lam-weighted error
 * of the coefficients C, else 0. fp32, ranks in order. */
int ora_keep_row(const float* C, const int8_t* codes, float scale, const float* lam, int r);

/* Eq. 9-12 on one Key token. cand receives the top-M ids in (d_Q, id) order. */
int ora_qsac_assign(const float* k, const float* mu, const float* w, int n_centroids,
                    int d, int group_size, int top_m, int* cand);

/* The same with the candidates ranked by the full quadratic form (ORA_METRIC_FULL):
 * e = k - mu_j (fp32), t_c = sum_c' m[c][c'] e_c' (c' in order), d_j = sum_c e_c t_c.
 * m is [d][d] fp32; the Eq. 12 score still uses w. */
int ora_qsac_assign_full(const float* k, const float* mu, const float* m, const float* w, int n_centroids,
                         int d, int group_size, int top_m, int* cand);

/* Plain nearest centroid (Euclidean), ties to the lower id. */
int ora_nearest(const float* x, const float* mu, int n_centroids, int d);

/* Eq. 6, Eq. 8 and Eq. 15, plus Lloyd K-means centroids (Eq. 3). m_out
 * [B,H,d,d] (optional) receives Mn = M / ((1/d) tr M) rounded to fp32 (the
 * identity at cold start), the matrix of ORA_METRIC_FULL. */
int ora_calibrate(const ora_cfg* cfg, const float* q_hist, long long n_hist,
                  const float* k_cal, const float* v_cal, long long n_cal, int kmeans_iters,
                  float* mu_k, float* mu_v, float* w, float* u_t, float* lam, float* m_out);

/* Cyclic Jacobi eigendecomposition of a symmetric n x n matrix (fp64).
 * Returns eigenvalues descending in lam and eigenvectors as rows of vecs_t. */
int ora_eigh(const double* a, int n, double* lam, double* vecs_t);

/* QSAC + INT2 residual + PSAC for Keys, nearest centroid + INT2 for Values,
 * written into cache slots [n_cached, n_cached + n_new) of every (b, h).
 * coef_f32 [B,H,n_new,r], k_ids/v_ids [B,H,n_new] and cand [B,H,n_new,M] are
 * optional diagnostics (NULL to skip). lam [B,H,r] (the stored eigenvalues) is
 * read only with ORA_STORE_GATE, m_full [B,H,d,d] only with ORA_METRIC_FULL. */
int ora_append(const ora_cfg* cfg, const float* mu_k, const float* mu_v, const float* w,
               const float* u_t, const float* lam, const float* m_full, uint8_t* cache, long long n_cached,
               const float* k_new, const float* v_new, long long n_new,
               float* coef_f32, int* k_ids, int* v_ids, int* cand);

/* App. D.1 per-chunk coefficient layout: the PSAC rows of slots [start, start + n)
 * of every (b, h) as one record, dense or sparse, whichever is smaller counting
 * the sparse indices. A row is kept when its FP16 scale is non-zero (a zero
 * scale means zero codes: the gate dropped it, or C was zero). Little-endian:
 *   header   16 B: u32 layout (0 dense, 1 sparse), u32 n, u32 r, u32 B*H
 *   dense    codes [BH][n][r] int8, then scales [BH][n] binary16
 *   sparse   counts [BH] u32, then for each (b, h) in order: indices [count] u16
 *            (slot - start, increasing), codes [count][r] int8, scales [count] binary16
 * Dense is 16 + BH n (r + 2) bytes, sparse 16 + 4 BH + (r + 4) x (kept rows);
 * sparse is taken only when strictly smaller. n <= 65536, r >= 1. */
#define ORA_COEF_DENSE 0
#define ORA_COEF_SPARSE 1
long long ora_coef_record_bytes(const ora_cfg* cfg, const uint8_t* cache, long long start, long long n, int* layout);
int ora_coef_pack(const ora_cfg* cfg, const uint8_t* cache, long long start, long long n, uint8_t* out,
                  long long out_bytes, long long* written);
/* Writes the record's rows back into slots [start, start + n) of every (b, h):
 * codes and scales, zeros for the rows a sparse record leaves out. */
int ora_coef_unpack(const ora_cfg* cfg, const uint8_t* rec, long long rec_bytes, uint8_t* cache, long long start,
                    long long n);

/* Decode slots [0, n) of head (b, h): Khat_0 (Eq. 4), INT8-decoded C, Vhat. */
int ora_decode(const ora_cfg* cfg, const float* mu_k, const float* mu_v,
               const uint8_t* cache, int b, int h, long long n,
               double* k0, double* chat, double* v);

/* Attention of selected Query rows over the packed cache (Eq. 5 with Eq. 17).
 * rows holds (b, h, i) triples. coef_override [B,H,n_cache,r] replaces the
 * decoded coefficients when non-NULL. logits [n_rows, n_cache] is optional and
 * holds -inf where a key is masked. A row with no visible key gets O = 0 and
 * lse = -inf. */
int ora_attend(const ora_cfg* cfg, const float* mu_k, const float* mu_v, const float* u_t,
               const uint8_t* cache, long long n_cache, const float* q, long long n_q,
               long long q_start, int frame_tokens, const float* coef_override,
               int n_rows, const int* rows, double* out, double* lse, double* logits);

/* The same over [packed history | active chunk]: keys [0, n_cache) decoded from
 * the cache, keys [n_cache, n_cache + n_act) taken exactly from k_act / v_act
 * ([B, n_act, H, d], rounded to the table type) with no PSAC term. Positions are
 * concatenated, so the mask and q_start (<= n_cache + n_act) refer to them. */
int ora_attend_active(const ora_cfg* cfg, const float* mu_k, const float* mu_v, const float* u_t,
                      const uint8_t* cache, long long n_cache, const float* k_act, const float* v_act,
                      long long n_act, const float* q, long long n_q, long long q_start, int frame_tokens,
                      const float* coef_override, int n_rows, const int* rows, double* out, double* lse,
                      double* logits);

/* The same with the packed keys in epochs: keys [epoch_start[e], epoch_start[e+1])
 * were appended with epoch e's tables ([n_epochs][B][H][...] for mu_k, mu_v,
 * u_t) and decode with them; their PSAC term uses q U_r of epoch e. */
int ora_attend_epochs(const ora_cfg* cfg, int n_epochs, const long long* epoch_start, const float* mu_k,
                      const float* mu_v, const float* u_t, const uint8_t* cache, long long n_cache,
                      const float* k_act, const float* v_act, long long n_act, const float* q, long long n_q,
                      long long q_start, int frame_tokens, const float* coef_override, int n_rows, const int* rows,
                      double* out, double* lse, double* logits);

int ora_max_threads(void);
void ora_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
