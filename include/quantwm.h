/*
 * quantwm.h: C ABI of libquantwm.so, the QuantWM hot path for AMD Instinct
 * MI355X (gfx950).
 *
 * QuantWM (arxiv 2609.26425) keeps the KV cache of a causal video world model
 * as BF16 centroids plus group-wise INT2 residuals (Eq. 3-4). Keys pick their
 * centroid by quantization-sensitivity-aware clustering (QSAC, Sec. 4.1,
 * Eq. 6-12). A low-rank compensation along the top historical Query directions
 * (PSAC, Sec. 4.2, Eq. 13-17) corrects the logits. Packed storage follows
 * App. D.1.
 *
 * Conventions for every entry point:
 *  - Pointers named *device* point to GPU memory that the caller allocated and
 *    owns. The library never allocates device memory and keeps no state between
 *    calls, except the per-thread message behind quantwm_last_error() and the
 *    static device buffer of quantwm_attend_noalloc (held per device).
 *  - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued
 *    asynchronously on it; outputs are valid once the stream has reached that
 *    point. Calls that touch the same buffers must be ordered on one stream.
 *  - Activations are contiguous token-major [B, N, H, d] tensors of the config's
 *    dtype (BF16 or FP32); all device pointers must be 16-byte aligned.
 *  - Arguments are validated on the host before anything is enqueued; a failed
 *    check returns a non-zero status, enqueues nothing, and sets the message.
 *    Non-finite inputs are outside the domain. A device fault surfaces at the
 *    caller's next synchronisation.
 */
#ifndef QUANTWM_H
#define QUANTWM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  QWM_OK = 0,
  QWM_ERR_INVALID_ARG = 1, /* null/misaligned pointer, negative size, bad range */
  QWM_ERR_UNSUPPORTED = 2, /* a shape the library has no kernel for */
  QWM_ERR_CAPACITY = 3,    /* tokens would exceed the cache capacity */
  QWM_ERR_HIP = 4          /* a HIP runtime call or a launch failed */
} quantwm_status;

typedef enum { QWM_F32 = 0, QWM_BF16 = 1 } quantwm_dtype;

typedef struct {
  int32_t batch;       /* B: independent rollouts */
  int32_t heads;       /* H */
  int32_t head_dim;    /* d: 64 or 128 */
  int32_t n_centroids; /* Kc in [1, 256]; ids are uint8 (App. D.1) */
  int32_t group_size;  /* G: INT2 residual group along channels; 16, 32 or 64, divides d */
  int32_t rank;        /* r: PSAC rank in [0, 32]; 0 disables PSAC (Eq. 16) */
  int32_t top_m;       /* M: QSAC candidates in [1, 8] (Sec. 4.1; the paper uses 4) */
  int32_t dtype;       /* quantwm_dtype of Q/K/V/O, centroids and U_r */
  int64_t capacity;    /* cache slots per (b, h), at most 2^26 */
  int32_t storage;     /* QWM_STORE_* flags, 0 for the plain format (App. D.1 options) */
  int32_t metric;      /* QWM_METRIC_*: distance of the QSAC candidate search */
  int64_t coef_rows;   /* QWM_STORE_SPARSE: PSAC rows in each (b, h) pool, 0 = one per slot */
  int64_t coef_stage;  /* QWM_STORE_SPARSE: staging rows, the largest n_new of one append call */
} quantwm_config;

/* QSAC candidate metric (quantwm_config.metric).
 * QWM_METRIC_DIAG (0): Eq. 9, sum_c w_c (k_c - mu_c)^2 with w from Eq. 8.
 * QWM_METRIC_FULL (1): the full quadratic form (k - mu)^T Mn (k - mu) of the
 *   diagonal-approximation ablation (App. C), with Mn = M / ((1/d) tr M) the
 *   Eq. 6 second moment over the mean of its diagonal (so diag(Mn) = w; the
 *   identity at cold start). Only the top-M candidate ranking changes: the
 *   Eq. 12 score, the quantisers and the cache format are those of
 *   QWM_METRIC_DIAG. The calibration block then carries Mn (field m). */
#define QWM_METRIC_DIAG 0
#define QWM_METRIC_FULL 1

/* Packed-storage options of App. D.1 (flags of quantwm_config.storage).
 * QWM_STORE_SCALE_I8: the Eq. 2 step sizes t_g of a token-head's groups are kept
 *   as 8-bit codes c_g = RN(t_g / sigma) in [0, 255] with one binary16 secondary
 *   scale sigma = RN16(max_g t_g / 255) per token-head; the step is sigma * c_g
 *   (exact in fp32), and the residual is quantised with it.
 * QWM_STORE_GATE: a PSAC row is kept only when its INT8 codes lower the
 *   Query-weighted error approximated on the principal subspace,
 *   sum_k lam_k (C_k - code_k * cscale)^2 < sum_k lam_k C_k^2 (fp32, ranks in
 *   order, lam from the calibration block); otherwise the row and its scale are
 *   stored as zeros.
 * Every attention call decodes both options, in every form (plain, key split,
 * active chunk in one launch or two parts, calibration epochs in one launch or
 * per epoch). */
#define QWM_STORE_SCALE_I8 1
#define QWM_STORE_GATE 2
/* QWM_STORE_SPARSE (needs rank >= 1 and coef_stage >= 1): the per-chunk choice
 * of App. D.1 between dense and sparse PSAC coefficient layouts, in the cache
 * that attention reads. The rows of each (b, h) live in a pool of coef_rows
 * rows, found through a directory with one 16-byte entry per 64-slot tile,
 * {u32 base, u32 0, u64 mask}: bit i of the mask says slot 64 T + i has a row,
 * at pool row base + (set bits below i); rows are in slot order. Each append
 * call is one chunk: per (b, h) it stores every row of the chunk (dense) or
 * only the rows with a non-zero scale (sparse), whichever is smaller counting
 * one mask bit per slot as the sparse index, sparse iff
 * kept (r + 2) + ceil(n / 8) < n (r + 2). A row with no room left in the pool
 * is not stored (it reads as a zero row, as a dropped one does) and is counted
 * (quantwm_coef_pool_usage). The chunk's rows are first written to staging
 * rows in the cache, so one append call takes at most coef_stage tokens
 * (QWM_ERR_CAPACITY otherwise). Attention reads rows through the directory in
 * every form except the logits hook and the chunk records (quantwm_coef_pack /
 * unpack), which read slot-addressed rows and refuse such a cache. */
#define QWM_STORE_SPARSE 4

/* ------------------------------------------------------------------ sizes */

/* Bytes of the packed K+V cache for cfg (0 if cfg is invalid). Layout: ten
 * sections, each starting on a 256-byte boundary, each [B*H][slots][bytes per
 * token] with slots = capacity rounded up to 64:
 *   K codes    d/4 bytes: channel c in bits 2(c%4) of byte c/4 (four INT2 codes per byte)
 *   K ids      1 byte: centroid id (uint8)
 *   K zp       ceil(d/G/4) bytes: group g in bits 2(g%4) of byte g/4 (INT2 zero-points)
 *   K scale    2*d/G bytes: IEEE binary16 group scales, little-endian
 *              (with QWM_STORE_SCALE_I8: d/G bytes, the 8-bit codes c_g)
 *   K coef     r bytes: INT8 PSAC coefficients
 *   K cscale   2 bytes (0 if r = 0): binary16 row scale of the coefficients
 *   V codes, V ids, V zp, V scale: as for K (Values carry no PSAC row).
 *   K sigma, V sigma  2 bytes each, only with QWM_STORE_SCALE_I8: the binary16
 *              secondary scale of the token-head's group scales.
 * With QWM_STORE_SPARSE the K coef and K cscale sections hold [B*H][coef_rows]
 * rows instead of one per slot, and four sections follow: the directory
 * [B*H][slots/64] of 16 bytes, the u32 overflow counters [B*H], and the staging
 * rows, codes [B*H][coef_stage][r] then binary16 scales [B*H][coef_stage].
 * A token's reconstruction is centroid + scale * (code - zero_point) (Eq. 4),
 * with scale = sigma * c_g under QWM_STORE_SCALE_I8, and its coefficients are
 * code * cscale (Eq. 16, App. D.1). */
size_t quantwm_cache_bytes(const quantwm_config* cfg);

/* Packed bytes per token-head for Keys and Values. Returns a status. */
quantwm_status quantwm_token_bytes(const quantwm_config* cfg, int32_t* k_bytes, int32_t* v_bytes);

/* Bytes of the calibration block: one slab per (b, h) of calib_slab_bytes. */
size_t quantwm_calib_bytes(const quantwm_config* cfg);

/* Byte offsets of the fields inside one (b, h) slab of the calibration block:
 *   mu_k, mu_v  [Kc][d] dtype   Key / Value centroids (Eq. 3)
 *   a_k         [Kc][d] f32     -2 * w_c * mu_k[j][c]   (search constants of Eq. 9;
 *                               with QWM_METRIC_FULL: -2 * p_jc, p_j = Mn mu_k[j])
 *   b_k         [Kc]    f32     sum_c w_c * mu_k[j][c]^2 (QWM_METRIC_FULL: sum_c p_jc mu_k[j][c])
 *   a_v, b_v                    the same for Values with w = 1
 *   w           [d]     f32     channel sensitivities (Eq. 8)
 *   wg          [d/G]   f32     per-group sums of w (Eq. 12)
 *   u_t         [r][d]  dtype   U_r transposed: row k is the k-th eigenvector (Eq. 15)
 *   lam         [r]     f32     the matching eigenvalues (0 at cold start)
 *   u_dr        [d][rs] f32     U_r itself (the transpose of u_t), ranks zero-padded to
 *                               rs = 16 (r <= 16) or 32 (r <= 32), for per-channel use
 *   m           [d][d]  f32     Mn, only with QWM_METRIC_FULL (no bytes otherwise)
 *   mu_k16, mu_v16 [Kc][d] binary16  BF16 configs only (no bytes otherwise): the
 *                               centroids times 2^-e_k (2^-e_v), e the exponent that puts
 *                               the table's largest magnitude in [2^14, 2^15) (0 for an
 *                               all-zero table), rounded to binary16: exact for every
 *                               component of at least 2^-31 times that largest one
 *   e16         [2]     int32   e_k, e_v (BF16 configs only)
 *   a_k3        [3][Kc][d] BF16  BF16 configs only: a_k split into three BF16 planes
 *                               whose sum is a_k exactly (the first two truncate, the
 *                               third is the exact remainder) for the matrix-core
 *                               Key search */
typedef struct {
  int64_t slab_bytes;
  int64_t mu_k, mu_v, a_k, b_k, a_v, b_v, w, wg, u_t, lam, u_dr, m, mu_k16, mu_v16, e16, a_k3;
} quantwm_calib_layout;
quantwm_status quantwm_calib_offsets(const quantwm_config* cfg, quantwm_calib_layout* out);

/* Device workspace bytes that quantwm_calibrate needs for these token counts. */
size_t quantwm_calibrate_workspace_bytes(const quantwm_config* cfg, int64_t n_hist, int64_t n_calib);

/* ------------------------------------------------------------ calibration */

/* Builds the calibration block from method-level tables (all device):
 * mu_k, mu_v [B,H,Kc,d] dtype; w [B,H,d] f32; u_t [B,H,r,d] dtype (NULL allowed
 * when r = 0); lam [B,H,r] f32 or NULL (then stored as 0); m [B,H,d,d] f32, the
 * matrix of QWM_METRIC_FULL (required with it, ignored otherwise). It derives
 * the search constants and group sums (Eq. 9 or the full form, Eq. 12) on the
 * device. */
quantwm_status quantwm_calib_pack(const quantwm_config* cfg, const void* mu_k, const void* mu_v,
                                  const float* w, const void* u_t, const float* lam, const float* m,
                                  void* calib, void* stream);

/* QSAC/PSAC statistics and centroids for every (b, h):
 *  - Eq. 6: M = (1/n_hist) sum q q^T over q_hist [B,n_hist,H,d] (fp64 on the device);
 *  - Eq. 8: w_c = M_cc / (tr(M)/d);
 *  - Eq. 15: U_r = top-r eigenvectors of M (host fp64 Jacobi; sorted by
 *    eigenvalue, each vector's largest-magnitude entry positive);
 *  - Eq. 3: centroids by deterministic Lloyd K-means (kmeans_iters rounds) on
 *    k_calib / v_calib [B,n_calib,H,d], starting from tokens floor(j*n/Kc).
 * n_hist == 0 is the cold start: w = 1 and U_r = 0, so PSAC stores zero rows.
 * Needs n_calib >= 1 and a device workspace of
 * quantwm_calibrate_workspace_bytes(). The call synchronises `stream` (it reads
 * M back to the host). */
quantwm_status quantwm_calibrate(const quantwm_config* cfg, const void* q_hist, int64_t n_hist,
                                 const void* k_calib, const void* v_calib, int64_t n_calib,
                                 int32_t kmeans_iters, void* calib, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Running Query statistics for calibration epochs (Eq. 6 computed online, the
 * streaming setting of Sec. 5 and App. C.3). A stats buffer holds a 256-byte
 * header (int64 token count) and the fp64 sums of q q^T, [B*H][d][d]. The caller
 * zeroes it once; a zero count is the cold start. */
size_t quantwm_stats_bytes(const quantwm_config* cfg);

/* Adds q q^T of the n Query tokens q [B,n,H,d] (dtype, device) to the sums and n
 * to the count. The sums continue from their stored values in token order, so
 * any sequence of updates equals one pass over all tokens in order. Ordered on
 * `stream` like every call; n == 0 is a no-op. */
quantwm_status quantwm_stats_update(const quantwm_config* cfg, const void* q, int64_t n, void* stats,
                                    void* stream);

/* quantwm_calibrate with the statistics of a stats buffer in place of q_hist:
 * M = sums / count (Eq. 6), w (Eq. 8), U_r (Eq. 15), and the centroids by
 * K-means on k_calib / v_calib (Eq. 3), e.g. the chunk that opens the epoch.
 * Workspace: quantwm_calibrate_workspace_bytes(cfg, 0, n_calib). Synchronises
 * `stream` (it reads the sums back to the host). */
quantwm_status quantwm_calibrate_epoch(const quantwm_config* cfg, const void* stats, const void* k_calib,
                                       const void* v_calib, int64_t n_calib, int32_t kmeans_iters, void* calib,
                                       void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------- hot path */

/* Quantize-on-append (Sec. 4.1-4.2, App. D.1) of n_new new tokens per (b, h)
 * into cache slots [n_cached, n_cached + n_new):
 *  - Keys: QSAC picks z = argmin of Eq. 12 over the top-M centroids by Eq. 9;
 *    the residual is quantised per group to INT2 with an FP16 scale and an INT2
 *    zero-point (Eq. 1-2, range extended to contain 0); PSAC stores
 *    C = (k - khat_0) U_r (Eq. 13, 16) as INT8 with an FP16 row scale.
 *  - Values: nearest centroid and the same INT2 residual, no PSAC.
 * The Eq. 9 search uses the expanded distance b_j + sum_c a_jc k_c in fp32.
 * With BF16 data it and the PSAC product run on matrix cores, with each fp32
 * operand split into three BF16 parts whose sum is exact: the products are
 * exact and only the order of the fp32 sums differs from a channel-order
 * evaluation, so a centroid id can differ from an exact-arithmetic choice only
 * where two distances tie to fp32 rounding. Integer decisions after the
 * search (Eq. 12 score, INT2 and INT8 codes) follow the equations' order in
 * fp32 with IEEE division and round-to-nearest-even.
 * k_new, v_new: [B,n_new,H,d] dtype. coef_f32_out: optional [B,H,n_new,r] f32
 * copy of C before INT8 rounding. n_new == 0 is a no-op. Needs
 * n_cached + n_new <= capacity; with BF16 data, ceil(n_new / 128) * B * H must
 * be below 2^24 (QWM_ERR_UNSUPPORTED otherwise). */
quantwm_status quantwm_append(const quantwm_config* cfg, const void* calib, void* cache,
                              int64_t n_cached, const void* k_new, const void* v_new,
                              int64_t n_new, float* coef_f32_out, void* stream);

/* Device workspace bytes that quantwm_attend can use for these sizes (0 when
 * it has no use for one). With it, a launch that would give the GPU fewer than
 * two workgroups per compute unit splits every Query block's key range over
 * several workgroups and merges their partial softmax results (the log-sum-exp
 * merge of Eq. 5 over disjoint key sets); the result is the same up to rounding.
 * The size depends on the current device's compute-unit count. */
size_t quantwm_attend_workspace_bytes(const quantwm_config* cfg, int64_t n_cache, int64_t n_q);

/* Attention of a Query chunk over the packed cache (Eq. 5 with Eq. 17):
 * L = (q . khat_0 + (q U_r) . chat) / sqrt(d), softmax over visible keys, times
 * vhat. Query i sits at absolute position q_start + i; key j is visible iff
 * j < q_start, or (j - q_start)/F <= i/F (block-causal by frames of
 * F = frame_tokens). q: [B,n_q,H,d] dtype; out: [B,n_q,H,d] dtype;
 * lse_out: optional [B,H,n_q] f32 natural-log sum-exp (-inf for a row with no
 * visible key, whose O is 0). Needs 0 <= q_start <= n_cache <= capacity.
 * n_q == 0 is a no-op. Keys and Values are dequantised in registers; the cache
 * is only ever read in packed form. workspace: optional device scratch of
 * workspace_bytes, 256-byte aligned, owned by the caller and not read back (NULL,
 * or fewer bytes than quantwm_attend_workspace_bytes(), means no split). Calls
 * that share a workspace must be ordered on one stream. QWM_ERR_UNSUPPORTED
 * when n_q or the key count (n_cache, plus n_act for the active-chunk forms)
 * exceeds 0x7fff0000 per head. */
quantwm_status quantwm_attend(const quantwm_config* cfg, const void* calib, const void* cache,
                              int64_t n_cache, const void* q, int64_t n_q, int64_t q_start,
                              int32_t frame_tokens, void* out, float* lse_out, void* workspace,
                              size_t workspace_bytes, void* stream);

/* quantwm_attend over [packed history | active chunk] (Sec. 5 streaming setting:
 * the chunk being generated stays in BF16 until it is complete and appended).
 * Keys [0, n_cache) come from the packed cache; keys [n_cache, n_cache + n_act)
 * are k_act / v_act ([B, n_act, H, d] dtype, device, 16-byte aligned), used
 * exactly, with no PSAC term. Positions are concatenated: the mask is that of
 * quantwm_attend over n_cache + n_act keys, and q_start <= n_cache + n_act.
 * n_act <= 2^26. With n_act == 0 this is quantwm_attend. With a workspace of
 * quantwm_attend_active_workspace_bytes(cfg, n_cache, n_act, n_q) bytes or more
 * (256-byte aligned) the call runs in two parts merged by log-sum-exp (the LSE
 * merge of the streaming setting): the packed keys of whole 64-key tiles
 * through the plain attention kernel, the remaining keys (the last packed tile
 * and the active chunk) through the general one. With a smaller workspace it
 * takes quantwm_attend_workspace_bytes(cfg, n_cache + n_act, n_q) as for
 * quantwm_attend, and NULL runs one launch. All forms give the same result up
 * to fp32 rounding order. */
quantwm_status quantwm_attend_active(const quantwm_config* cfg, const void* calib, const void* cache,
                                     int64_t n_cache, const void* k_act, const void* v_act, int64_t n_act,
                                     const void* q, int64_t n_q, int64_t q_start, int32_t frame_tokens,
                                     void* out, float* lse_out, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* Workspace bytes for quantwm_attend_active: the larger of the two-part form's
 * (two or more fp32 partial planes; none without an active chunk or with fewer
 * than 64 packed keys) and the split workspace of
 * quantwm_attend_workspace_bytes(cfg, n_cache + n_act, n_q). */
size_t quantwm_attend_active_workspace_bytes(const quantwm_config* cfg, int64_t n_cache, int64_t n_act,
                                             int64_t n_q);

/* quantwm_attend_active over a cache appended in calibration epochs (the
 * streaming setting of Sec. 5: statistics and centroids are refreshed at chunk
 * boundaries, and every chunk keeps the tables it was quantised with). Packed
 * keys [epoch_start[e], epoch_start[e+1]) were appended with calibration block e
 * of `calibs` (n_epochs blocks of quantwm_calib_bytes(cfg), contiguous, device);
 * they decode with that block's centroids, and their PSAC term is
 * (q U_r^(e)) . c with that block's U_r (Eq. 17 per epoch). epoch_start is a
 * host array: epoch_start[0] = 0, each epoch spans at least 64 keys, every start
 * is < n_cache; n_epochs in [1, 64]. n_epochs == 1 is quantwm_attend_active. */
quantwm_status quantwm_attend_epochs(const quantwm_config* cfg, const void* calibs, int32_t n_epochs,
                                     const int64_t* epoch_start, const void* cache, int64_t n_cache,
                                     const void* k_act, const void* v_act, int64_t n_act, const void* q,
                                     int64_t n_q, int64_t q_start, int32_t frame_tokens, void* out,
                                     float* lse_out, void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes for the per-epoch form of quantwm_attend_epochs (n_epochs >=
 * 2; 0 otherwise): each
 * epoch's packed keys run through the plain attention kernel with that epoch's
 * calibration block as partial results of their own; with an active chunk, the
 * last whole packed tile on runs through the general kernel; everything merges
 * by log-sum-exp. epoch_start is the host array of the call. Given at least
 * this much (256-byte aligned) the call takes that form; otherwise the
 * one-launch form, with the split workspace of
 * quantwm_attend_workspace_bytes(cfg, n_cache + n_act, n_q). Both give the same
 * result up to fp32 rounding order. */
size_t quantwm_attend_epochs_workspace_bytes(const quantwm_config* cfg, int32_t n_epochs,
                                             const int64_t* epoch_start, int64_t n_cache, int64_t n_act,
                                             int64_t n_q);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): quantwm_attend with
 * no workspace argument. Where quantwm_attend would split the key range
 * (launches of fewer than two workgroups per compute unit), the partial
 * results go to a static device buffer of QWM_ATTEND_NOALLOC_SCRATCH_BYTES that
 * the library holds on each device it runs on until the process ends; the
 * split count is cut to what the buffer holds. The call allocates nothing
 * (its first call on a device only looks up that device's buffer address).
 * Arguments, layouts and results are those of quantwm_attend (equal up to fp32
 * rounding order; bit-equal when the split count is the same). Calls on one
 * device share the buffer: calls that overlap in time on one device (different
 * streams, or host threads) race and give undefined results; calls ordered on
 * one stream are safe. Nothing in the buffer needs clearing between calls.
 * QWM_ERR_CAPACITY when even a two-way split does not fit (B*H*n_q*(d + 2)*8
 * bytes above the buffer); quantwm_attend with a caller workspace takes such
 * sizes. On a 256-CU device the split rule never asks for that: a launch large
 * enough to need it has two workgroups per CU and does not split. */
#define QWM_ATTEND_NOALLOC_SCRATCH_BYTES (128u << 20)
quantwm_status quantwm_attend_noalloc(const quantwm_config* cfg, const void* calib, const void* cache,
                                      int64_t n_cache, const void* q, int64_t n_q, int64_t q_start,
                                      int32_t frame_tokens, void* out, float* lse_out, void* stream);

/* Test hook: the scaled logits of quantwm_attend, [B,H,n_q,n_cache] f32,
 * -inf where masked. Same tile code as quantwm_attend. Query i is chunk row
 * q_first + i (absolute position q_start + q_first + i): key j is visible iff
 * j < q_start or (j - q_start)/F <= (q_first + i)/F, so rows of any frame can
 * be checked without the rows before them. q_first = 0 is the Query chunk of
 * quantwm_attend. Needs q_first >= 0. */
quantwm_status quantwm_logits(const quantwm_config* cfg, const void* calib, const void* cache,
                              int64_t n_cache, const void* q, int64_t n_q, int64_t q_start, int64_t q_first,
                              int32_t frame_tokens, float* logits_out, void* stream);

/* ------------------------------------------- per-chunk coefficient records */

/* App. D.1 per-chunk choice between dense and sparse PSAC coefficient layouts,
 * for a chunk of the cache moved out of it (offloaded to the host, written to
 * disk, sent elsewhere): the INT8 rows and FP16 scales of slots
 * [start, start + n) of every (b, h) as one record, dense or sparse, whichever
 * is smaller counting the sparse indices. A row is kept when its scale is
 * non-zero; a zero scale means zero codes (the QWM_STORE_GATE rule dropped the
 * row, or its coefficients were zero), so the sparse form loses nothing. The
 * attention calls read the dense rows in the cache. Record (little-endian):
 *   header   16 B: u32 layout (QWM_COEF_DENSE or QWM_COEF_SPARSE), u32 n,
 *            u32 r, u32 B*H
 *   dense    codes [B*H][n][r] int8, then scales [B*H][n] binary16:
 *            16 + B*H*n*(r + 2) bytes
 *   sparse   counts [B*H] u32, then per (b, h) in order: indices [count] u16
 *            (slot - start, increasing), codes [count][r] int8, scales
 *            [count] binary16: 16 + 4*B*H + (r + 4) * (kept rows) bytes
 * Sparse is taken only when strictly smaller. Needs rank >= 1, 0 <= n <= 65536
 * and start + n <= capacity (QWM_ERR_INVALID_ARG otherwise). */
#define QWM_COEF_DENSE 0
#define QWM_COEF_SPARSE 1

/* Bytes a record buffer for n tokens must hold (the dense size, and at least
 * the header and counts); 0 if the arguments are invalid. */
size_t quantwm_coef_record_max_bytes(const quantwm_config* cfg, int64_t n);

/* Writes the record of the chunk into `record` (device, record_bytes >=
 * quantwm_coef_record_max_bytes(cfg, n)); *written (host) receives its size and
 * *layout (host, may be NULL) the layout chosen. The cache is only read. The
 * call synchronises `stream` once, to read the kept-row counts; the record is
 * complete when the stream reaches the call's last kernel. */
quantwm_status quantwm_coef_pack(const quantwm_config* cfg, const void* cache, int64_t start, int64_t n,
                                 void* record, size_t record_bytes, int64_t* written, int32_t* layout,
                                 void* stream);

/* Writes a record made by quantwm_coef_pack back into slots [start, start + n)
 * of every (b, h): the codes and scales of its rows, and zeros for the rows a
 * sparse record leaves out. Nothing else in the cache changes. The header and
 * counts are read back and checked first (n, r and B*H must match the call,
 * and record_bytes must cover the record), which synchronises `stream`. */
quantwm_status quantwm_coef_unpack(const quantwm_config* cfg, const void* record, size_t record_bytes,
                                   void* cache, int64_t start, int64_t n, void* stream);

/* QWM_STORE_SPARSE: PSAC rows held by the pools for cache slots [0, n_cache)
 * summed over every (b, h) (*rows_used), and rows that found no room in a pool
 * since the cache was zeroed (*rows_dropped); host outputs. Synchronises
 * `stream` (it reads the directory back). */
quantwm_status quantwm_coef_pool_usage(const quantwm_config* cfg, const void* cache, int64_t n_cache,
                                       int64_t* rows_used, int64_t* rows_dropped, void* stream);

/* Message for the last non-OK status on the calling thread ("" if none). */
const char* quantwm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
