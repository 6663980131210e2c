// Shared host/device definitions of the QuantWM HIP library: packed-cache and
// calibration-block layouts, element types and kernel argument blocks.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/quantwm.h"

namespace qwm {

typedef __bf16 bf16;

// Packed cache layout (App. D.1 storage, section order fixed by quantwm.h).
struct CacheLayout {
  int d, ng, zpb, r;
  int i8;  // group scales as 8-bit codes + a binary16 secondary scale per token
  int sb;  // group-scale bytes per token: 2 ng (binary16) or ng (8-bit codes)
  int k_bytes, v_bytes;
  int64_t slots;  // per (b, h): capacity rounded up to 64
  int64_t k_codes, k_ids, k_zp, k_scale, k_coef, k_cscale;
  int64_t v_codes, v_ids, v_zp, v_scale;
  int64_t k_sigma, v_sigma;  // i8 only: the secondary scale per token
  int sparse;                // PSAC rows in a pool per (b, h), found through a tile directory
  int64_t pool, stage;       // rows per (b, h) in the coefficient sections and in the staging rows
  int64_t k_dir, k_over, k_st_codes, k_st_scale;  // sparse only
  int64_t total;
};

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

inline CacheLayout cache_layout(const quantwm_config& c) {
  CacheLayout L;
  L.d = c.head_dim;
  L.ng = c.head_dim / c.group_size;
  L.zpb = (L.ng + 3) / 4;
  L.r = c.rank;
  L.slots = (c.capacity + 63) / 64 * 64;
  L.i8 = (c.storage & QWM_STORE_SCALE_I8) != 0;
  L.sb = L.i8 ? L.ng : 2 * L.ng;
  L.sparse = (c.storage & QWM_STORE_SPARSE) != 0;
  L.pool = L.sparse && c.coef_rows > 0 ? c.coef_rows : L.slots;
  L.stage = L.sparse ? c.coef_stage : 0;
  const int64_t bh = int64_t(c.batch) * c.heads, rows = bh * L.slots;
  int64_t at = 0;
  auto take_n = [&](int64_t n, int64_t per) { int64_t o = at; at = align256(at + n * per); return o; };
  auto take = [&](int64_t per_token) { return take_n(rows, per_token); };
  L.k_codes = take(L.d / 4);
  L.k_ids = take(1);
  L.k_zp = take(L.zpb);
  L.k_scale = take(L.sb);
  L.k_coef = take_n(bh * L.pool, L.r);
  L.k_cscale = take_n(bh * L.pool, L.r > 0 ? 2 : 0);
  L.v_codes = take(L.d / 4);
  L.v_ids = take(1);
  L.v_zp = take(L.zpb);
  L.v_scale = take(L.sb);
  L.k_sigma = take(L.i8 ? 2 : 0);
  L.v_sigma = take(L.i8 ? 2 : 0);
  L.k_dir = take_n(bh * (L.slots / 64), L.sparse ? 16 : 0);
  L.k_over = take_n(bh, L.sparse ? 4 : 0);
  L.k_st_codes = take_n(bh * L.stage, L.r);
  L.k_st_scale = take_n(bh * L.stage, 2);
  L.total = at;
  L.v_bytes = L.d / 4 + 1 + L.zpb + L.sb + (L.i8 ? 2 : 0);
  L.k_bytes = L.v_bytes + (L.r > 0 ? L.r + 2 : 0);
  return L;
}

inline int elem_bytes(const quantwm_config& c) { return c.dtype == QWM_BF16 ? 2 : 4; }

// Row stride of the [d][rs] copy of U_r: ranks padded with zeros to 16 or 32.
inline int rank_stride(const quantwm_config& c) { return c.rank == 0 ? 0 : (c.rank <= 16 ? 16 : 32); }

inline quantwm_calib_layout calib_layout(const quantwm_config& c) {
  quantwm_calib_layout L;
  const int64_t d = c.head_dim, K = c.n_centroids, r = c.rank, e = elem_bytes(c);
  int64_t at = 0;
  auto take = [&](int64_t bytes) { int64_t o = at; at = align256(at + bytes); return o; };
  L.mu_k = take(K * d * e);
  L.mu_v = take(K * d * e);
  L.a_k = take(K * d * 4);
  L.b_k = take(K * 4);
  L.a_v = take(K * d * 4);
  L.b_v = take(K * 4);
  L.w = take(d * 4);
  L.wg = take((d / c.group_size) * 4);
  L.u_t = take(r * d * e);
  L.lam = take(r * 4);
  L.u_dr = take(int64_t(rank_stride(c)) * d * 4);
  L.m = take(c.metric == QWM_METRIC_FULL ? d * d * 4 : 0);
  const bool h16 = c.dtype == QWM_BF16;  // binary16 copies for the attention producers
  L.mu_k16 = take(h16 ? K * d * 2 : 0);
  L.mu_v16 = take(h16 ? K * d * 2 : 0);
  L.e16 = take(h16 ? 8 : 0);
  L.a_k3 = take(h16 ? 3 * K * d * 2 : 0);
  L.slab_bytes = at;
  return L;
}

// ------------------------------------------------------------ kernel args

struct AppendArgs {
  const uint8_t* calib;
  int64_t slab;
  int64_t o_mu_k, o_mu_v, o_a_k, o_b_k, o_a_v, o_b_v, o_wg, o_u_t, o_u_dr;
  int64_t o_a_k3;  // BF16 configs: the three BF16 planes of a_k
  uint8_t* cache;
  CacheLayout L;
  const void* k;
  const void* v;
  int64_t n_new, n_cached;
  int heads, n_centroids, rank, top_m;
  float* coef_out;
  int gate;        // QWM_STORE_GATE with r > 0
  int64_t o_lam;   // eigenvalues in the slab (read with the gate)
};

constexpr int kMaxEpochs = 64;

struct AttendArgs {
  const uint8_t* calib;
  int64_t slab;
  int64_t o_mu_k, o_mu_v, o_u_t;
  int64_t o_mu_k16, o_mu_v16, o_e16;  // binary16 table copies and their exponents (BF16 configs)
  const uint8_t* cache;
  CacheLayout L;
  const void* q;
  void* out;
  float* lse;
  float* logits;
  int64_t n_cache, n_q, q_start;
  const void* k_act;  // [B, n_act, H, d] exact active-chunk Keys (after the packed ones)
  const void* v_act;
  int64_t n_act;
  int frame_tokens, heads, n_centroids, rank;
  int tables_in_lds;
  int n_split;    // workgroups per Query block, each over its share of the key tiles
  // calibration epochs: packed keys [epoch_start[e], epoch_start[e+1]) were
  // appended with the calibration block at calib + e * calib_stride
  int n_epochs;
  int64_t calib_stride;
  int64_t epoch_start[64];
  float* part_o;  // [n_split][B*H][n_q][d] unnormalised partial outputs (n_split > 1)
  float* part_ml; // [n_split][B*H][n_q][2] running max (raw logits) and sum per partial
  // a launch that covers key tiles [tile_lo, ...) only and writes its partial
  // results at planes split_base + split; the caller merges them (partial = 1)
  int64_t tile_lo;
  int split_base;
  int partial;
  int64_t key_lo;  // keys below are masked (a launch over one calibration epoch's keys)
  int64_t q_row0;  // logits hook only: chunk row of the first Query (frame count of the mask)
};

// keys per attention tile
constexpr int kAttendTileKeys = 64;

// Launchers. Append: one translation unit per (element type, head_dim, group
// size); fp32 Keys and Values on the vector ALU, BF16 ones with the centroid
// searches on the matrix cores.
template <int D, int G>
hipError_t launch_append_f32(const AppendArgs& a, int batch, hipStream_t s);
template <int D, int G>
hipError_t launch_append_bf16(const AppendArgs& a, int batch, hipStream_t s);
hipError_t launch_attend_f32(const AttendArgs& a, int d, int batch, bool logits, hipStream_t s);
hipError_t launch_attend_bf16(const AttendArgs& a, int d, int batch, bool logits, hipStream_t s);
size_t attend_lds_bytes(int d, int elem, int rank, int n_centroids, bool tables_in_lds);
int attend_splits(int64_t n_q, int heads, int batch, int64_t n_cache, int cus);
bool attend_tables_fit(int d, int elem, int rank, int n_centroids);

hipError_t launch_derive_constants(const quantwm_config& c, uint8_t* calib, hipStream_t s);
hipError_t launch_pack_tables(const quantwm_config& c, const void* mu_k, const void* mu_v,
                              const float* w, const void* u_t, const float* lam, const float* m,
                              uint8_t* calib, hipStream_t s);
hipError_t launch_moment_accumulate(const quantwm_config& c, const void* q, int64_t n, double* sums, int64_t* count,
                                    hipStream_t s);
hipError_t launch_second_moment(const quantwm_config& c, const void* q, int64_t n, double* m_out,
                                hipStream_t s);
hipError_t launch_attend_combine(const AttendArgs& a, int d, int batch, bool is_bf16, hipStream_t s);
hipError_t launch_coef_count(const quantwm_config& c, const void* cache, int64_t start, int n, void* counts,
                             hipStream_t s);
hipError_t launch_coef_pack(const quantwm_config& c, const void* cache, int64_t start, int n, void* record,
                            int layout, hipStream_t s);
hipError_t launch_coef_unpack(const quantwm_config& c, const void* record, int layout, void* cache, int64_t start,
                              int n, hipStream_t s);
// QWM_STORE_SPARSE: stores one append call's staged rows into the pools and the directory
hipError_t launch_coef_commit(const quantwm_config& c, void* cache, int64_t n_cached, int64_t n, hipStream_t s);
hipError_t launch_kmeans(const quantwm_config& c, const void* x, int64_t n, int iters, uint8_t* calib,
                         int64_t o_mu, int32_t* assign_ws, hipStream_t s);

// Host fp64 symmetric eigensolver: eigenvalues descending, eigenvectors as rows.
void host_eigh(const double* a, int n, double* lam, double* vecs_t);

}  // namespace qwm
