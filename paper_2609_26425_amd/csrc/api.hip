// C ABI of libquantwm.so: host-side validation, size queries and launches.
// Every check runs before anything is enqueued; nothing here allocates device
// memory.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "qwm_common.h"

namespace {
// largest Query or key count per head the attention kernels take (positions
// are 32-bit there, with room for a tile past the end)
constexpr int64_t kMaxPositions = 0x7fff0000;

thread_local std::string g_error;

quantwm_status fail(quantwm_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
quantwm_status fail(quantwm_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return s;
}

quantwm_status ok() {
  g_error.clear();
  return QWM_OK;
}

quantwm_status hip_fail(hipError_t e, const char* what) {
  return fail(QWM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Shape support of the library; INVALID for nonsense, UNSUPPORTED for shapes
// that are meaningful but have no kernel here.
quantwm_status check_cfg(const quantwm_config* c) {
  if (!c) return fail(QWM_ERR_INVALID_ARG, "config is null");
  if (c->batch < 1 || c->heads < 1) return fail(QWM_ERR_INVALID_ARG, "batch and heads must be >= 1");
  if (c->head_dim < 1 || c->group_size < 1 || c->head_dim % c->group_size)
    return fail(QWM_ERR_INVALID_ARG, "group_size must divide head_dim");
  if (c->n_centroids < 1 || c->n_centroids > 256)
    return fail(QWM_ERR_INVALID_ARG, "n_centroids must be in [1, 256] (uint8 ids)");
  if (c->rank < 0 || c->rank > c->head_dim) return fail(QWM_ERR_INVALID_ARG, "rank must be in [0, head_dim]");
  if (c->top_m < 1) return fail(QWM_ERR_INVALID_ARG, "top_m must be >= 1");
  if (c->capacity < 0) return fail(QWM_ERR_INVALID_ARG, "capacity must be >= 0");
  if (c->dtype != QWM_F32 && c->dtype != QWM_BF16) return fail(QWM_ERR_INVALID_ARG, "dtype must be F32 or BF16");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(QWM_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (c->group_size != 16 && c->group_size != 32 && c->group_size != 64)
    return fail(QWM_ERR_UNSUPPORTED, "group_size must be 16, 32 or 64");
  if (c->rank > 32) return fail(QWM_ERR_UNSUPPORTED, "rank must be <= 32");
  if (c->top_m > 8) return fail(QWM_ERR_UNSUPPORTED, "top_m must be <= 8");
  if (c->capacity > (int64_t(1) << 26))  // kernels address a head's slots with 32-bit offsets
    return fail(QWM_ERR_UNSUPPORTED, "capacity must be <= 2^26 slots per (b, h)");
  if (c->storage & ~(QWM_STORE_SCALE_I8 | QWM_STORE_GATE | QWM_STORE_SPARSE))
    return fail(QWM_ERR_INVALID_ARG, "storage has unknown flags 0x%x", unsigned(c->storage));
  if (c->storage & QWM_STORE_SPARSE) {
    if (c->rank < 1) return fail(QWM_ERR_INVALID_ARG, "QWM_STORE_SPARSE needs PSAC rows (rank >= 1)");
    if (c->coef_rows < 0 || c->coef_rows > (int64_t(1) << 26))
      return fail(QWM_ERR_INVALID_ARG, "coef_rows must be in [0, 2^26]");
    if (c->coef_stage < 1 || c->coef_stage > (int64_t(1) << 26))
      return fail(QWM_ERR_INVALID_ARG, "QWM_STORE_SPARSE needs coef_stage in [1, 2^26]");
  }
  if (c->metric != QWM_METRIC_DIAG && c->metric != QWM_METRIC_FULL)
    return fail(QWM_ERR_INVALID_ARG, "metric must be QWM_METRIC_DIAG or QWM_METRIC_FULL");
  return QWM_OK;
}

quantwm_status check_dev(const void* p, const char* name, bool required = true) {
  if (!p) return required ? fail(QWM_ERR_INVALID_ARG, "%s is null", name) : QWM_OK;
  if (!aligned16(p)) return fail(QWM_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return QWM_OK;
}

template <typename T, int D>
hipError_t launch_append_td(const qwm::AppendArgs& a, int g, int batch, hipStream_t s) {
  constexpr bool bf = sizeof(T) == 2;
  if (g == 16) return bf ? qwm::launch_append_bf16<D, 16>(a, batch, s) : qwm::launch_append_f32<D, 16>(a, batch, s);
  if (g == 32) return bf ? qwm::launch_append_bf16<D, 32>(a, batch, s) : qwm::launch_append_f32<D, 32>(a, batch, s);
  if (g == 64) return bf ? qwm::launch_append_bf16<D, 64>(a, batch, s) : qwm::launch_append_f32<D, 64>(a, batch, s);
  return hipErrorInvalidValue;
}

#define QWM_TRY(x)                         \
  do {                                     \
    quantwm_status _s = (x);               \
    if (_s != QWM_OK) return _s;           \
  } while (0)

}  // namespace

extern "C" {

const char* quantwm_last_error(void) { return g_error.c_str(); }

}  // extern "C"

namespace {
// shape checks shared by the coefficient-record calls
quantwm_status check_coef(const quantwm_config* cfg, int64_t start, int64_t n) {
  QWM_TRY(check_cfg(cfg));
  if (cfg->rank < 1) return fail(QWM_ERR_INVALID_ARG, "the config has no PSAC rows (rank 0)");
  if (cfg->storage & QWM_STORE_SPARSE)
    return fail(QWM_ERR_INVALID_ARG, "chunk records read slot-addressed rows; the cache keeps sparse rows");
  if (start < 0 || n < 0 || n > 65536 || start + n > cfg->capacity)
    return fail(QWM_ERR_INVALID_ARG, "need start >= 0, 0 <= n <= 65536 and start + n <= capacity");
  return QWM_OK;
}
int64_t coef_dense_bytes(const quantwm_config* c, int64_t n) {
  return 16 + int64_t(c->batch) * c->heads * n * (c->rank + 2);
}
}  // namespace

extern "C" {

size_t quantwm_coef_record_max_bytes(const quantwm_config* cfg, int64_t n) {
  if (check_cfg(cfg) != QWM_OK || cfg->rank < 1 || n < 0 || n > 65536) return 0;
  const int64_t floor = 16 + 4 * int64_t(cfg->batch) * cfg->heads, dense = coef_dense_bytes(cfg, n);
  return size_t(dense > floor ? dense : floor);
}

quantwm_status quantwm_coef_pack(const quantwm_config* cfg, const void* cache, int64_t start, int64_t n,
                                 void* record, size_t record_bytes, int64_t* written, int32_t* layout,
                                 void* stream) {
  QWM_TRY(check_coef(cfg, start, n));
  QWM_TRY(check_dev(cache, "cache"));
  QWM_TRY(check_dev(record, "record"));
  if (!written) return fail(QWM_ERR_INVALID_ARG, "written is null");
  const size_t need = quantwm_coef_record_max_bytes(cfg, n);
  if (record_bytes < need) return fail(QWM_ERR_INVALID_ARG, "record buffer too small: %zu < %zu bytes", record_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t nbh = int64_t(cfg->batch) * cfg->heads;
  hipError_t he;
  // kept-row counts go where a sparse record keeps them
  uint8_t* rec = static_cast<uint8_t*>(record);
  if ((he = qwm::launch_coef_count(*cfg, cache, start, int(n), rec + 16, s)) != hipSuccess)
    return hip_fail(he, "coef count launch");
  std::vector<uint32_t> counts(static_cast<size_t>(nbh));
  if ((he = hipMemcpyAsync(counts.data(), rec + 16, counts.size() * 4, hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (he = hipStreamSynchronize(s)) != hipSuccess)
    return hip_fail(he, "coef count readback");
  int64_t kept = 0;
  for (uint32_t k : counts) kept += k;
  const int64_t dense = coef_dense_bytes(cfg, n), sparse = 16 + 4 * nbh + kept * (cfg->rank + 4);
  const int lay = sparse < dense ? QWM_COEF_SPARSE : QWM_COEF_DENSE;
  if ((he = qwm::launch_coef_pack(*cfg, cache, start, int(n), record, lay, s)) != hipSuccess)
    return hip_fail(he, "coef pack launch");
  *written = lay == QWM_COEF_SPARSE ? sparse : dense;
  if (layout) *layout = lay;
  return ok();
}

quantwm_status quantwm_coef_unpack(const quantwm_config* cfg, const void* record, size_t record_bytes,
                                   void* cache, int64_t start, int64_t n, void* stream) {
  QWM_TRY(check_coef(cfg, start, n));
  QWM_TRY(check_dev(record, "record"));
  QWM_TRY(check_dev(cache, "cache"));
  if (record_bytes < 16) return fail(QWM_ERR_INVALID_ARG, "record shorter than its header");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t nbh = int64_t(cfg->batch) * cfg->heads;
  hipError_t he;
  uint32_t hdr[4];
  if ((he = hipMemcpyAsync(hdr, record, 16, hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (he = hipStreamSynchronize(s)) != hipSuccess)
    return hip_fail(he, "coef header readback");
  if (hdr[1] != uint32_t(n) || hdr[2] != uint32_t(cfg->rank) || int64_t(hdr[3]) != nbh)
    return fail(QWM_ERR_INVALID_ARG, "record header (n %u, r %u, heads %u) does not match the call", hdr[1], hdr[2],
                hdr[3]);
  if (hdr[0] == QWM_COEF_DENSE) {
    if (int64_t(record_bytes) < coef_dense_bytes(cfg, n)) return fail(QWM_ERR_INVALID_ARG, "dense record is truncated");
  } else if (hdr[0] == QWM_COEF_SPARSE) {
    if (int64_t(record_bytes) < 16 + 4 * nbh) return fail(QWM_ERR_INVALID_ARG, "sparse record is truncated");
    std::vector<uint32_t> counts(static_cast<size_t>(nbh));
    if ((he = hipMemcpyAsync(counts.data(), static_cast<const uint8_t*>(record) + 16, counts.size() * 4,
                             hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (he = hipStreamSynchronize(s)) != hipSuccess)
      return hip_fail(he, "coef counts readback");
    int64_t total = 16 + 4 * nbh;
    for (uint32_t k : counts) {
      if (int64_t(k) > n) return fail(QWM_ERR_INVALID_ARG, "sparse record counts more rows than the chunk holds");
      total += int64_t(k) * (cfg->rank + 4);
    }
    if (int64_t(record_bytes) < total) return fail(QWM_ERR_INVALID_ARG, "sparse record is truncated");
  } else {
    return fail(QWM_ERR_INVALID_ARG, "record layout %u is neither dense nor sparse", hdr[0]);
  }
  if ((he = qwm::launch_coef_unpack(*cfg, record, int(hdr[0]), cache, start, int(n), s)) != hipSuccess)
    return hip_fail(he, "coef unpack launch");
  return ok();
}

size_t quantwm_cache_bytes(const quantwm_config* cfg) {
  if (check_cfg(cfg) != QWM_OK) return 0;
  return size_t(qwm::cache_layout(*cfg).total);
}

quantwm_status quantwm_token_bytes(const quantwm_config* cfg, int32_t* k_bytes, int32_t* v_bytes) {
  QWM_TRY(check_cfg(cfg));
  if (!k_bytes || !v_bytes) return fail(QWM_ERR_INVALID_ARG, "output pointer is null");
  const qwm::CacheLayout L = qwm::cache_layout(*cfg);
  *k_bytes = L.k_bytes;
  *v_bytes = L.v_bytes;
  return ok();
}

size_t quantwm_calib_bytes(const quantwm_config* cfg) {
  if (check_cfg(cfg) != QWM_OK) return 0;
  return size_t(qwm::calib_layout(*cfg).slab_bytes) * cfg->batch * cfg->heads;
}

quantwm_status quantwm_calib_offsets(const quantwm_config* cfg, quantwm_calib_layout* out) {
  QWM_TRY(check_cfg(cfg));
  if (!out) return fail(QWM_ERR_INVALID_ARG, "output pointer is null");
  *out = qwm::calib_layout(*cfg);
  return ok();
}

size_t quantwm_calibrate_workspace_bytes(const quantwm_config* cfg, int64_t n_hist, int64_t n_calib) {
  if (check_cfg(cfg) != QWM_OK || n_hist < 0 || n_calib < 0) return 0;
  const size_t bh = size_t(cfg->batch) * cfg->heads, d = cfg->head_dim;
  const size_t m = qwm::align256(int64_t(bh * d * d * sizeof(double)));
  const size_t as = qwm::align256(int64_t(bh * size_t(n_calib) * sizeof(int32_t)));
  return m + as;
}

quantwm_status quantwm_calib_pack(const quantwm_config* cfg, const void* mu_k, const void* mu_v, const float* w,
                                  const void* u_t, const float* lam, const float* m, void* calib, void* stream) {
  QWM_TRY(check_cfg(cfg));
  QWM_TRY(check_dev(mu_k, "mu_k"));
  QWM_TRY(check_dev(mu_v, "mu_v"));
  QWM_TRY(check_dev(w, "w"));
  QWM_TRY(check_dev(u_t, "u_t", false));
  QWM_TRY(check_dev(lam, "lam", false));
  const bool full = cfg->metric == QWM_METRIC_FULL;
  QWM_TRY(check_dev(m, "m", full));
  QWM_TRY(check_dev(calib, "calib"));
  if (cfg->rank > 0 && !u_t) return fail(QWM_ERR_INVALID_ARG, "u_t is null with rank > 0");
  const hipError_t e = qwm::launch_pack_tables(*cfg, mu_k, mu_v, w, u_t, lam, full ? m : nullptr,
                                               static_cast<uint8_t*>(calib), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "calib_pack launch");
  return ok();
}

// Eq. 8 and Eq. 15 on the host in fp64 from the second moment M ([B*H][d][d],
// already divided by the token count), then Eq. 3 centroids on the device.
// cold: no historical Query yet (w = 1, U_r = 0).
static quantwm_status finish_calibration(const quantwm_config& c, const std::vector<double>& M, bool cold,
                                         const void* k_calib, const void* v_calib, int64_t n_calib,
                                         int32_t kmeans_iters, uint8_t* cal, int32_t* assign, hipStream_t s) {
  const quantwm_calib_layout C = qwm::calib_layout(c);
  const int bh = c.batch * c.heads, d = c.head_dim, r = c.rank, e = qwm::elem_bytes(c);
  hipError_t he;
  std::vector<float> w(size_t(bh) * d), lam(size_t(bh) * (r > 0 ? r : 1));
  std::vector<uint8_t> ut(size_t(bh) * (r > 0 ? r : 1) * d * e, 0);
  std::vector<double> ev(d), vt(size_t(d) * d);
  const bool full = c.metric == QWM_METRIC_FULL;
  std::vector<float> mn(full ? size_t(bh) * d * d : 0);
  for (int i = 0; i < bh; ++i) {
    const double* Mi = M.data() + size_t(i) * d * d;
    double tr = 0.0;
    for (int k = 0; k < d; ++k) tr += Mi[size_t(k) * d + k];
    float* wi = w.data() + size_t(i) * d;
    float* mi = full ? mn.data() + size_t(i) * d * d : nullptr;
    if (cold || tr == 0.0) {  // cold start: uniform sensitivity, PSAC inactive
      for (int k = 0; k < d; ++k) wi[k] = 1.0f;
      for (int k = 0; k < r; ++k) lam[size_t(i) * r + k] = 0.0f;
      if (mi)
        for (int k = 0; k < d * d; ++k) mi[k] = (k / d == k % d) ? 1.0f : 0.0f;
      continue;
    }
    for (int k = 0; k < d; ++k) wi[k] = (float)(Mi[size_t(k) * d + k] / (tr / (double)d));
    // the full metric: M over the mean of its diagonal (its diagonal is w)
    if (mi)
      for (int k = 0; k < d * d; ++k) mi[k] = (float)(Mi[k] / (tr / (double)d));
    qwm::host_eigh(Mi, d, ev.data(), vt.data());
    for (int k = 0; k < r; ++k) {
      lam[size_t(i) * r + k] = (float)ev[k];
      for (int cc = 0; cc < d; ++cc) {
        const double x = vt[size_t(k) * d + cc];
        uint8_t* dst = ut.data() + ((size_t(i) * r + k) * d + cc) * e;
        if (e == 4) {
          const float f = (float)x;
          std::memcpy(dst, &f, 4);
        } else {  // bf16, one rounding from fp64 (nearest, ties to even)
          uint64_t u;
          std::memcpy(&u, &x, 8);
          u += ((uint64_t(1) << 44) - 1) + ((u >> 45) & 1);
          u &= ~((uint64_t(1) << 45) - 1);
          double y;
          std::memcpy(&y, &u, 8);
          const float f = (float)y;
          uint32_t fb;
          std::memcpy(&fb, &f, 4);
          const uint16_t hb = uint16_t(fb >> 16);
          std::memcpy(dst, &hb, 2);
        }
      }
    }
  }
  auto put = [&](int64_t off, const void* src, size_t row) -> hipError_t {
    if (row == 0) return hipSuccess;
    return hipMemcpy2DAsync(cal + off, size_t(C.slab_bytes), src, row, row, size_t(bh), hipMemcpyHostToDevice, s);
  };
  if ((he = put(C.w, w.data(), size_t(d) * 4)) != hipSuccess) return hip_fail(he, "w upload");
  if (full && (he = put(C.m, mn.data(), size_t(d) * d * 4)) != hipSuccess) return hip_fail(he, "m upload");
  if (r > 0) {
    if ((he = put(C.u_t, ut.data(), size_t(r) * d * e)) != hipSuccess) return hip_fail(he, "u_t upload");
    if ((he = put(C.lam, lam.data(), size_t(r) * 4)) != hipSuccess) return hip_fail(he, "lam upload");
  }
  // Eq. 3: Key and Value centroids by Lloyd K-means on the calibration tokens.
  if ((he = qwm::launch_kmeans(c, k_calib, n_calib, kmeans_iters, cal, C.mu_k, assign, s)) != hipSuccess)
    return hip_fail(he, "kmeans (K)");
  if ((he = qwm::launch_kmeans(c, v_calib, n_calib, kmeans_iters, cal, C.mu_v, assign, s)) != hipSuccess)
    return hip_fail(he, "kmeans (V)");
  if ((he = qwm::launch_derive_constants(c, cal, s)) != hipSuccess) return hip_fail(he, "derive");
  // the host staging buffers die with this call
  if ((he = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(he, "calibrate sync");
  return ok();
}

quantwm_status quantwm_calibrate(const quantwm_config* cfg, const void* q_hist, int64_t n_hist, const void* k_calib,
                                 const void* v_calib, int64_t n_calib, int32_t kmeans_iters, void* calib,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  QWM_TRY(check_cfg(cfg));
  if (n_hist < 0 || n_calib < 1 || kmeans_iters < 0)
    return fail(QWM_ERR_INVALID_ARG, "need n_hist >= 0, n_calib >= 1, kmeans_iters >= 0");
  QWM_TRY(check_dev(q_hist, "q_hist", n_hist > 0));
  QWM_TRY(check_dev(k_calib, "k_calib"));
  QWM_TRY(check_dev(v_calib, "v_calib"));
  QWM_TRY(check_dev(calib, "calib"));
  QWM_TRY(check_dev(workspace, "workspace"));
  if (workspace_bytes < quantwm_calibrate_workspace_bytes(cfg, n_hist, n_calib))
    return fail(QWM_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes,
                quantwm_calibrate_workspace_bytes(cfg, n_hist, n_calib));
  const quantwm_config& c = *cfg;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int bh = c.batch * c.heads, d = c.head_dim;
  double* m_dev = static_cast<double*>(workspace);
  int32_t* assign = reinterpret_cast<int32_t*>(static_cast<uint8_t*>(workspace) +
                                               qwm::align256(int64_t(size_t(bh) * d * d * sizeof(double))));
  hipError_t he;
  // Eq. 6 on the device
  std::vector<double> M(size_t(bh) * d * d, 0.0);
  if (n_hist > 0) {
    if ((he = qwm::launch_second_moment(c, q_hist, n_hist, m_dev, s)) != hipSuccess) return hip_fail(he, "moment");
    if ((he = hipMemcpyAsync(M.data(), m_dev, M.size() * sizeof(double), hipMemcpyDeviceToHost, s)) != hipSuccess)
      return hip_fail(he, "moment readback");
    if ((he = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(he, "moment sync");
  }
  return finish_calibration(c, M, n_hist == 0, k_calib, v_calib, n_calib, kmeans_iters, static_cast<uint8_t*>(calib),
                            assign, s);
}

size_t quantwm_stats_bytes(const quantwm_config* cfg) {
  if (check_cfg(cfg) != QWM_OK) return 0;
  return 256 + size_t(cfg->batch) * cfg->heads * cfg->head_dim * cfg->head_dim * sizeof(double);
}

quantwm_status quantwm_stats_update(const quantwm_config* cfg, const void* q, int64_t n, void* stats, void* stream) {
  QWM_TRY(check_cfg(cfg));
  if (n < 0) return fail(QWM_ERR_INVALID_ARG, "n must be >= 0");
  if (n == 0) return ok();
  QWM_TRY(check_dev(q, "q"));
  QWM_TRY(check_dev(stats, "stats"));
  int64_t* count = static_cast<int64_t*>(stats);
  double* sums = reinterpret_cast<double*>(static_cast<uint8_t*>(stats) + 256);
  const hipError_t he = qwm::launch_moment_accumulate(*cfg, q, n, sums, count, static_cast<hipStream_t>(stream));
  if (he != hipSuccess) return hip_fail(he, "stats update");
  return ok();
}

quantwm_status quantwm_calibrate_epoch(const quantwm_config* cfg, const void* stats, const void* k_calib,
                                       const void* v_calib, int64_t n_calib, int32_t kmeans_iters, void* calib,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  QWM_TRY(check_cfg(cfg));
  if (n_calib < 1 || kmeans_iters < 0) return fail(QWM_ERR_INVALID_ARG, "need n_calib >= 1, kmeans_iters >= 0");
  QWM_TRY(check_dev(stats, "stats"));
  QWM_TRY(check_dev(k_calib, "k_calib"));
  QWM_TRY(check_dev(v_calib, "v_calib"));
  QWM_TRY(check_dev(calib, "calib"));
  QWM_TRY(check_dev(workspace, "workspace"));
  if (workspace_bytes < quantwm_calibrate_workspace_bytes(cfg, 0, n_calib))
    return fail(QWM_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes,
                quantwm_calibrate_workspace_bytes(cfg, 0, n_calib));
  const quantwm_config& c = *cfg;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t nm = size_t(c.batch) * c.heads * c.head_dim * c.head_dim;
  std::vector<double> M(nm);
  int64_t count = 0;
  hipError_t he;
  if ((he = hipMemcpyAsync(&count, stats, sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
      (he = hipMemcpyAsync(M.data(), static_cast<const uint8_t*>(stats) + 256, nm * sizeof(double),
                           hipMemcpyDeviceToHost, s)) != hipSuccess)
    return hip_fail(he, "stats readback");
  if ((he = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(he, "stats sync");
  if (count < 0) return fail(QWM_ERR_INVALID_ARG, "stats count is negative (buffer not initialised?)");
  // Eq. 6: M = sum / count, the same fp64 division as the one-pass moment
  if (count > 0)
    for (double& x : M) x = x / (double)count;
  return finish_calibration(c, M, count == 0, k_calib, v_calib, n_calib, kmeans_iters, static_cast<uint8_t*>(calib),
                            static_cast<int32_t*>(workspace), s);
}

quantwm_status quantwm_append(const quantwm_config* cfg, const void* calib, void* cache, int64_t n_cached,
                              const void* k_new, const void* v_new, int64_t n_new, float* coef_f32_out,
                              void* stream) {
  QWM_TRY(check_cfg(cfg));
  if (n_cached < 0 || n_new < 0) return fail(QWM_ERR_INVALID_ARG, "token counts must be >= 0");
  if (n_cached + n_new > cfg->capacity)
    return fail(QWM_ERR_CAPACITY, "n_cached + n_new = %lld exceeds capacity %lld", (long long)(n_cached + n_new),
                (long long)cfg->capacity);
  if (n_new == 0) return ok();
  if ((cfg->storage & QWM_STORE_SPARSE) && n_new > cfg->coef_stage)
    return fail(QWM_ERR_CAPACITY, "n_new = %lld exceeds the %lld staging rows of a sparse-row cache (coef_stage)",
                (long long)n_new, (long long)cfg->coef_stage);
  QWM_TRY(check_dev(calib, "calib"));
  QWM_TRY(check_dev(cache, "cache"));
  QWM_TRY(check_dev(k_new, "k_new"));
  QWM_TRY(check_dev(v_new, "v_new"));
  if (coef_f32_out && (reinterpret_cast<uintptr_t>(coef_f32_out) & 3))
    return fail(QWM_ERR_INVALID_ARG, "coef_f32_out is not 4-byte aligned");
  if (n_new > (int64_t(1) << 31) - 256) return fail(QWM_ERR_UNSUPPORTED, "n_new too large for one call");
  if (cfg->dtype == QWM_BF16 && (n_new + 127) / 128 * cfg->heads * cfg->batch >= (int64_t(1) << 24))
    return fail(QWM_ERR_UNSUPPORTED, "ceil(n_new / 128) * heads * batch must be below 2^24 (one launch)");
  const quantwm_calib_layout C = qwm::calib_layout(*cfg);
  qwm::AppendArgs a;
  a.calib = static_cast<const uint8_t*>(calib);
  a.slab = C.slab_bytes;
  a.o_mu_k = C.mu_k; a.o_mu_v = C.mu_v; a.o_a_k = C.a_k; a.o_b_k = C.b_k;
  a.o_a_v = C.a_v; a.o_b_v = C.b_v; a.o_wg = C.wg; a.o_u_t = C.u_t; a.o_u_dr = C.u_dr; a.o_a_k3 = C.a_k3;
  a.o_lam = C.lam;
  a.gate = (cfg->storage & QWM_STORE_GATE) && cfg->rank > 0 ? 1 : 0;
  a.cache = static_cast<uint8_t*>(cache);
  a.L = qwm::cache_layout(*cfg);
  a.k = k_new; a.v = v_new;
  a.n_new = n_new; a.n_cached = n_cached;
  a.heads = cfg->heads; a.n_centroids = cfg->n_centroids; a.rank = cfg->rank; a.top_m = cfg->top_m;
  a.coef_out = coef_f32_out;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  const bool bf = cfg->dtype == QWM_BF16;
  if (cfg->head_dim == 64) e = bf ? launch_append_td<qwm::bf16, 64>(a, cfg->group_size, cfg->batch, s)
                                  : launch_append_td<float, 64>(a, cfg->group_size, cfg->batch, s);
  else e = bf ? launch_append_td<qwm::bf16, 128>(a, cfg->group_size, cfg->batch, s)
              : launch_append_td<float, 128>(a, cfg->group_size, cfg->batch, s);
  if (e != hipSuccess) return hip_fail(e, "append launch");
  if (cfg->storage & QWM_STORE_SPARSE) {
    if ((e = qwm::launch_coef_commit(*cfg, cache, n_cached, n_new, s)) != hipSuccess)
      return hip_fail(e, "sparse-row commit launch");
  }
  return ok();
}

// Scratch of quantwm_attend_noalloc: the partial-result planes of its key
// split. Each device holds its own copy while the library is loaded. Host code
// never passes the array's name to a kernel (on the host it is only a
// stand-in): it takes the device address from hipGetSymbolAddress, once per
// device, and uses that.
static __device__ __align__(256) unsigned char scratch[QWM_ATTEND_NOALLOC_SCRATCH_BYTES];

static constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];

static quantwm_status noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(QWM_ERR_UNSUPPORTED, "device %d above the %d the library tracks", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "scratch address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return QWM_OK;
}

// Compute units of the current device (256 on MI355X; 256 when no device answers,
// so that sizes agree between a host-only query and the launch).
static int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  return cus;
}

static size_t attend_split_bytes(const quantwm_config* cfg, int64_t n_cache, int64_t n_q, int* splits) {
  const int ns = qwm::attend_splits(n_q, cfg->heads, cfg->batch, n_cache, device_cus());
  if (splits) *splits = ns;
  if (ns <= 1) return 0;
  const size_t rows = size_t(ns) * cfg->batch * cfg->heads * size_t(n_q);
  const size_t o_bytes = (rows * cfg->head_dim * 4 + 255) / 256 * 256;
  return o_bytes + rows * 2 * 4;
}

size_t quantwm_attend_workspace_bytes(const quantwm_config* cfg, int64_t n_cache, int64_t n_q) {
  if (check_cfg(cfg) != QWM_OK || n_cache < 0 || n_q <= 0) return 0;
  return attend_split_bytes(cfg, n_cache, n_q, nullptr);
}

// Two-part form of the active-chunk call: the plain kernel over the packed keys
// of whole tiles [0, 64 floor(n_cache / 64)) as ns_a partial planes (its own key
// split), then the general kernel over the rest (one plane), then the merge.
static size_t active_two_part_bytes(const quantwm_config* cfg, int64_t n_cache, int64_t n_act, int64_t n_q,
                                    int* ns_a) {
  const int64_t nfl = n_cache / qwm::kAttendTileKeys * qwm::kAttendTileKeys;
  if (nfl == 0 || n_act == 0 || n_q <= 0) return 0;
  const int ns = qwm::attend_splits(n_q, cfg->heads, cfg->batch, nfl, device_cus());
  if (ns_a) *ns_a = ns;
  const size_t rows = size_t(ns + 1) * cfg->batch * cfg->heads * size_t(n_q);
  return (rows * cfg->head_dim * 4 + 255) / 256 * 256 + rows * 2 * 4;
}

// Per-epoch form of the epochs call: the keys of each calibration epoch through
// the plain kernel with that epoch's block (its own key split), then, with an
// active chunk, the general kernel from the last whole packed tile on; the
// partial planes merge by log-sum-exp. Ranges and plane counts per epoch.
struct EpochPlan {
  int n = 0, planes = 0;
  int64_t lo[qwm::kMaxEpochs], hi[qwm::kMaxEpochs];
  int ns[qwm::kMaxEpochs];
  int64_t tail_tile = -1;  // first tile of the general launch (active chunk), -1 if none
};

static EpochPlan plan_epochs(const quantwm_config* cfg, int n_epochs, const int64_t* es, int64_t n_cache,
                             int64_t n_act, int64_t n_q) {
  EpochPlan p;
  const int64_t kt = qwm::kAttendTileKeys;
  const int64_t end = n_act > 0 ? n_cache / kt * kt : n_cache;
  const int cus = device_cus();
  for (int e = 0; e < n_epochs; ++e) {
    const int64_t lo = es[e], hi0 = e + 1 < n_epochs ? es[e + 1] : n_cache, hi = hi0 < end ? hi0 : end;
    if (hi <= lo) continue;
    p.lo[p.n] = lo;
    p.hi[p.n] = hi;
    p.ns[p.n] = qwm::attend_splits(n_q, cfg->heads, cfg->batch, hi - lo, cus);
    p.planes += p.ns[p.n];
    ++p.n;
  }
  if (n_act > 0) {
    p.tail_tile = end / kt;
    p.planes += 1;
  }
  return p;
}

static size_t planes_bytes(const quantwm_config* cfg, int planes, int64_t n_q) {
  const size_t rows = size_t(planes) * cfg->batch * cfg->heads * size_t(n_q);
  return (rows * cfg->head_dim * 4 + 255) / 256 * 256 + rows * 2 * 4;
}

size_t quantwm_attend_epochs_workspace_bytes(const quantwm_config* cfg, int32_t n_epochs, const int64_t* epoch_start,
                                             int64_t n_cache, int64_t n_act, int64_t n_q) {
  if (check_cfg(cfg) != QWM_OK || n_cache < 0 || n_act < 0 || n_q <= 0) return 0;
  if (n_epochs < 2 || n_epochs > qwm::kMaxEpochs || !epoch_start) return 0;
  const EpochPlan p = plan_epochs(cfg, n_epochs, epoch_start, n_cache, n_act, n_q);
  const size_t per = planes_bytes(cfg, p.planes, n_q);
  const size_t split = attend_split_bytes(cfg, n_cache + n_act, n_q, nullptr);
  return per > split ? per : split;
}

size_t quantwm_attend_active_workspace_bytes(const quantwm_config* cfg, int64_t n_cache, int64_t n_act,
                                             int64_t n_q) {
  if (check_cfg(cfg) != QWM_OK || n_cache < 0 || n_act < 0 || n_q <= 0) return 0;
  const size_t two = active_two_part_bytes(cfg, n_cache, n_act, n_q, nullptr);
  const size_t split = attend_split_bytes(cfg, n_cache + n_act, n_q, nullptr);
  return two > split ? two : split;
}

// split_cap > 0 limits the key split of the plain form to that many parts.
static quantwm_status attend_common(const quantwm_config* cfg, const void* calib, int32_t n_epochs,
                                    const int64_t* epoch_start, const void* cache, int64_t n_cache,
                                    const void* k_act, const void* v_act, int64_t n_act, const void* q, int64_t n_q,
                                    int64_t q_start, int32_t frame_tokens, void* out, float* lse_out,
                                    float* logits_out, void* workspace, size_t workspace_bytes, void* stream,
                                    int split_cap = 0, int64_t q_first = 0) {
  QWM_TRY(check_cfg(cfg));
  if (n_epochs < 1 || n_epochs > qwm::kMaxEpochs) return fail(QWM_ERR_UNSUPPORTED, "n_epochs must be in [1, 64]");
  if (n_epochs > 1) {
    if (!epoch_start) return fail(QWM_ERR_INVALID_ARG, "epoch_start is null");
    if (epoch_start[0] != 0) return fail(QWM_ERR_INVALID_ARG, "epoch_start[0] must be 0");
    for (int e = 1; e < n_epochs; ++e) {
      if (epoch_start[e] - epoch_start[e - 1] < 64)
        return fail(QWM_ERR_INVALID_ARG, "epoch %d spans fewer than 64 keys", e - 1);
      if (epoch_start[e] >= n_cache) return fail(QWM_ERR_INVALID_ARG, "epoch %d starts at or past n_cache", e);
    }
  }
  if (n_cache < 0 || n_act < 0 || n_q < 0 || q_start < 0) return fail(QWM_ERR_INVALID_ARG, "sizes must be >= 0");
  if (n_cache > cfg->capacity) return fail(QWM_ERR_CAPACITY, "n_cache exceeds capacity");
  if (n_act > (int64_t(1) << 26)) return fail(QWM_ERR_UNSUPPORTED, "n_act above 2^26");
  if (q_start > n_cache + n_act) return fail(QWM_ERR_INVALID_ARG, "q_start > n_cache + n_act");
  if (frame_tokens < 1) return fail(QWM_ERR_INVALID_ARG, "frame_tokens must be >= 1");
  if (n_q == 0) return ok();
  QWM_TRY(check_dev(calib, "calib"));
  QWM_TRY(check_dev(cache, "cache"));
  QWM_TRY(check_dev(q, "q"));
  if (n_act > 0) {
    QWM_TRY(check_dev(k_act, "k_act"));
    QWM_TRY(check_dev(v_act, "v_act"));
  }
  if (logits_out) {
    if (reinterpret_cast<uintptr_t>(logits_out) & 3) return fail(QWM_ERR_INVALID_ARG, "logits_out misaligned");
  } else {
    QWM_TRY(check_dev(out, "out"));
    if (lse_out && (reinterpret_cast<uintptr_t>(lse_out) & 3)) return fail(QWM_ERR_INVALID_ARG, "lse_out misaligned");
  }
  if ((n_q + 255) / 256 > 0x7fffffff) return fail(QWM_ERR_UNSUPPORTED, "n_q too large");
  const bool sparse_rows = (cfg->storage & QWM_STORE_SPARSE) != 0;
  if (sparse_rows && logits_out)
    return fail(QWM_ERR_UNSUPPORTED, "the logits hook reads slot-addressed rows; the cache keeps sparse rows");
  const int elem = qwm::elem_bytes(*cfg);
  const bool tables = qwm::attend_tables_fit(cfg->head_dim, elem, cfg->rank, cfg->n_centroids);
  const quantwm_calib_layout C = qwm::calib_layout(*cfg);
  qwm::AttendArgs a;
  a.calib = static_cast<const uint8_t*>(calib);
  a.slab = C.slab_bytes;
  a.o_mu_k = C.mu_k; a.o_mu_v = C.mu_v; a.o_u_t = C.u_t;
  a.o_mu_k16 = C.mu_k16; a.o_mu_v16 = C.mu_v16; a.o_e16 = C.e16;
  a.cache = static_cast<const uint8_t*>(cache);
  a.L = qwm::cache_layout(*cfg);
  a.q = q; a.out = out; a.lse = lse_out; a.logits = logits_out;
  a.n_cache = n_cache; a.n_q = n_q; a.q_start = q_start;
  a.n_epochs = n_epochs;
  a.calib_stride = n_epochs > 1 ? int64_t(quantwm_calib_bytes(cfg)) : 0;
  for (int e = 0; e < qwm::kMaxEpochs; ++e) a.epoch_start[e] = e < n_epochs && n_epochs > 1 ? epoch_start[e] : 0;
  a.k_act = n_act > 0 ? k_act : nullptr;
  a.v_act = n_act > 0 ? v_act : nullptr;
  a.n_act = n_act;
  a.frame_tokens = frame_tokens; a.heads = cfg->heads; a.n_centroids = cfg->n_centroids; a.rank = cfg->rank;
  a.tables_in_lds = tables ? 1 : 0;
  a.n_split = 1;
  a.part_o = nullptr;
  a.part_ml = nullptr;
  if (!logits_out && workspace) {
    if (reinterpret_cast<uintptr_t>(workspace) & 255) return fail(QWM_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    int ns = 1;
    size_t need = attend_split_bytes(cfg, n_cache + n_act, n_q, &ns);
    if (split_cap > 0 && ns > split_cap) {
      ns = split_cap;
      need = planes_bytes(cfg, ns, n_q);
    }
    if (ns > 1 && workspace_bytes >= need) {
      const size_t rows = size_t(ns) * cfg->batch * cfg->heads * size_t(n_q);
      a.n_split = ns;
      a.part_o = static_cast<float*>(workspace);
      a.part_ml = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + (rows * cfg->head_dim * 4 + 255) / 256 * 256);
    }
  }
  a.tile_lo = 0;
  a.split_base = 0;
  a.partial = 0;
  a.key_lo = 0;
  a.q_row0 = logits_out ? q_first : 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // calibration epochs one by one through the plain kernel when the workspace
  // holds a partial plane per launch
  if (!logits_out && workspace && n_epochs > 1 && !sparse_rows) {
    const EpochPlan p = plan_epochs(cfg, n_epochs, epoch_start, n_cache, n_act, n_q);
    const size_t need = planes_bytes(cfg, p.planes, n_q);
    if (workspace_bytes >= need && p.planes > 0) {
      if (n_q > kMaxPositions || n_cache + n_act > kMaxPositions)
        return fail(QWM_ERR_UNSUPPORTED, "more than %lld Queries or keys per head", (long long)kMaxPositions);
      const size_t rows = size_t(p.planes) * cfg->batch * cfg->heads * size_t(n_q);
      a.part_o = static_cast<float*>(workspace);
      a.part_ml = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + (rows * cfg->head_dim * 4 + 255) / 256 * 256);
      const bool bf = cfg->dtype == QWM_BF16;
      auto run = [&](const qwm::AttendArgs& x) {
        return bf ? qwm::launch_attend_bf16(x, cfg->head_dim, cfg->batch, false, s)
                  : qwm::launch_attend_f32(x, cfg->head_dim, cfg->batch, false, s);
      };
      hipError_t e = hipSuccess;
      int base = 0;
      for (int i = 0; i < p.n && e == hipSuccess; ++i) {
        qwm::AttendArgs ea = a;  // one epoch's keys [lo, hi) with its own block
        const int ep = [&] {
          int k = 0;
          while (k + 1 < n_epochs && epoch_start[k + 1] <= p.lo[i]) ++k;
          return k;
        }();
        ea.calib = a.calib + int64_t(ep) * a.calib_stride;
        ea.n_epochs = 1;
        for (int k = 0; k < qwm::kMaxEpochs; ++k) ea.epoch_start[k] = 0;
        ea.n_cache = p.hi[i];
        ea.k_act = ea.v_act = nullptr;
        ea.n_act = 0;
        ea.tile_lo = p.lo[i] / qwm::kAttendTileKeys;
        ea.key_lo = p.lo[i];
        ea.n_split = p.ns[i];
        ea.split_base = base;
        ea.partial = 1;
        if ((n_q + 255) / 256 * int64_t(ea.n_split) > 0x7fffffff) return fail(QWM_ERR_UNSUPPORTED, "n_q too large");
        e = run(ea);
        base += p.ns[i];
      }
      if (e == hipSuccess && p.tail_tile >= 0) {
        qwm::AttendArgs ga = a;  // the last packed tile and the active chunk, all epochs
        ga.tile_lo = p.tail_tile;
        ga.n_split = 1;
        ga.split_base = base;
        ga.partial = 1;
        e = run(ga);
      }
      if (e == hipSuccess) {
        qwm::AttendArgs ca = a;
        ca.n_split = p.planes;
        e = qwm::launch_attend_combine(ca, cfg->head_dim, cfg->batch, bf, s);
      }
      if (e != hipSuccess) return hip_fail(e, "attend launch (per epoch)");
      return ok();
    }
  }
  // the active chunk in two parts when the workspace holds their partials: the
  // packed keys of whole tiles through the plain kernel, the rest through the
  // general one, merged by log-sum-exp
  int ns_a = 1;
  const size_t two = (!logits_out && workspace && n_act > 0 && n_epochs == 1 && !sparse_rows)
                         ? active_two_part_bytes(cfg, n_cache, n_act, n_q, &ns_a) : 0;
  const bool two_part = two > 0 && workspace_bytes >= two;
  if (two_part) {
    const size_t rows = size_t(ns_a + 1) * cfg->batch * cfg->heads * size_t(n_q);
    a.n_split = 1;
    a.part_o = static_cast<float*>(workspace);
    a.part_ml = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + (rows * cfg->head_dim * 4 + 255) / 256 * 256);
    if ((n_q + 255) / 256 * int64_t(ns_a) > 0x7fffffff) return fail(QWM_ERR_UNSUPPORTED, "n_q too large");
  }
  if ((n_q + 255) / 256 * int64_t(a.n_split) > 0x7fffffff) return fail(QWM_ERR_UNSUPPORTED, "n_q too large");
  // the kernel keeps Query and key positions in 32 bits
  if (n_q > kMaxPositions || n_cache + n_act > kMaxPositions)
    return fail(QWM_ERR_UNSUPPORTED, "more than %lld Queries or keys per head", (long long)kMaxPositions);
  const bool lg = logits_out != nullptr;
  if (two_part) {
    const bool bf = cfg->dtype == QWM_BF16;
    const int64_t nfl = n_cache / qwm::kAttendTileKeys * qwm::kAttendTileKeys;
    qwm::AttendArgs pa = a;  // packed part: keys [0, nfl) only, planes [0, ns_a)
    pa.n_cache = nfl;
    pa.k_act = pa.v_act = nullptr;
    pa.n_act = 0;
    pa.n_split = ns_a;
    pa.partial = 1;
    qwm::AttendArgs ga = a;  // the rest: tiles from nfl / 64 on, plane ns_a
    ga.tile_lo = nfl / qwm::kAttendTileKeys;
    ga.split_base = ns_a;
    ga.partial = 1;
    hipError_t e = bf ? qwm::launch_attend_bf16(pa, cfg->head_dim, cfg->batch, false, s)
                      : qwm::launch_attend_f32(pa, cfg->head_dim, cfg->batch, false, s);
    if (e == hipSuccess)
      e = bf ? qwm::launch_attend_bf16(ga, cfg->head_dim, cfg->batch, false, s)
             : qwm::launch_attend_f32(ga, cfg->head_dim, cfg->batch, false, s);
    if (e == hipSuccess) {
      qwm::AttendArgs ca = a;
      ca.n_split = ns_a + 1;
      e = qwm::launch_attend_combine(ca, cfg->head_dim, cfg->batch, bf, s);
    }
    if (e != hipSuccess) return hip_fail(e, "attend launch (two parts)");
    return ok();
  }
  const hipError_t e = cfg->dtype == QWM_BF16 ? qwm::launch_attend_bf16(a, cfg->head_dim, cfg->batch, lg, s)
                                              : qwm::launch_attend_f32(a, cfg->head_dim, cfg->batch, lg, s);
  if (e != hipSuccess) return hip_fail(e, "attend launch");
  return ok();
}

quantwm_status quantwm_attend(const quantwm_config* cfg, const void* calib, const void* cache, int64_t n_cache,
                              const void* q, int64_t n_q, int64_t q_start, int32_t frame_tokens, void* out,
                              float* lse_out, void* workspace, size_t workspace_bytes, void* stream) {
  return attend_common(cfg, calib, 1, nullptr, cache, n_cache, nullptr, nullptr, 0, q, n_q, q_start, frame_tokens, out,
                       lse_out, nullptr, workspace, workspace_bytes, stream);
}

quantwm_status quantwm_attend_active(const quantwm_config* cfg, const void* calib, const void* cache,
                                     int64_t n_cache, const void* k_act, const void* v_act, int64_t n_act,
                                     const void* q, int64_t n_q, int64_t q_start, int32_t frame_tokens, void* out,
                                     float* lse_out, void* workspace, size_t workspace_bytes, void* stream) {
  return attend_common(cfg, calib, 1, nullptr, cache, n_cache, k_act, v_act, n_act, q, n_q, q_start, frame_tokens, out,
                       lse_out, nullptr, workspace, workspace_bytes, stream);
}

quantwm_status quantwm_attend_epochs(const quantwm_config* cfg, const void* calibs, int32_t n_epochs,
                                     const int64_t* epoch_start, const void* cache, int64_t n_cache,
                                     const void* k_act, const void* v_act, int64_t n_act, const void* q, int64_t n_q,
                                     int64_t q_start, int32_t frame_tokens, void* out, float* lse_out,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  return attend_common(cfg, calibs, n_epochs, epoch_start, cache, n_cache, k_act, v_act, n_act, q, n_q, q_start,
                       frame_tokens, out, lse_out, nullptr, workspace, workspace_bytes, stream);
}

quantwm_status quantwm_attend_noalloc(const quantwm_config* cfg, const void* calib, const void* cache,
                                      int64_t n_cache, const void* q, int64_t n_q, int64_t q_start,
                                      int32_t frame_tokens, void* out, float* lse_out, void* stream) {
  QWM_TRY(check_cfg(cfg));
  if (n_cache < 0 || n_q < 0) return fail(QWM_ERR_INVALID_ARG, "sizes must be >= 0");
  // the key split quantwm_attend would take, cut to what the static buffer holds
  int ns = 1;
  if (n_q > 0) (void)attend_split_bytes(cfg, n_cache, n_q, &ns);
  void* scratch = nullptr;
  if (ns > 1) {
    while (ns > 1 && planes_bytes(cfg, ns, n_q) > QWM_ATTEND_NOALLOC_SCRATCH_BYTES) --ns;
    if (ns < 2)
      return fail(QWM_ERR_CAPACITY,
                  "the key split of this call needs %zu bytes of scratch for two parts; the static buffer of "
                  "quantwm_attend_noalloc holds %zu (quantwm_attend with a workspace takes any size)",
                  planes_bytes(cfg, 2, n_q), size_t(QWM_ATTEND_NOALLOC_SCRATCH_BYTES));
    QWM_TRY(noalloc_scratch(&scratch));
  }
  return attend_common(cfg, calib, 1, nullptr, cache, n_cache, nullptr, nullptr, 0, q, n_q, q_start, frame_tokens,
                       out, lse_out, nullptr, scratch, scratch ? size_t(QWM_ATTEND_NOALLOC_SCRATCH_BYTES) : 0, stream,
                       ns);
}

quantwm_status quantwm_coef_pool_usage(const quantwm_config* cfg, const void* cache, int64_t n_cache,
                                       int64_t* rows_used, int64_t* rows_dropped, void* stream) {
  QWM_TRY(check_cfg(cfg));
  if (!(cfg->storage & QWM_STORE_SPARSE)) return fail(QWM_ERR_INVALID_ARG, "the config keeps no sparse rows");
  if (n_cache < 0 || n_cache > cfg->capacity) return fail(QWM_ERR_INVALID_ARG, "need 0 <= n_cache <= capacity");
  if (!rows_used || !rows_dropped) return fail(QWM_ERR_INVALID_ARG, "output pointer is null");
  QWM_TRY(check_dev(cache, "cache"));
  const qwm::CacheLayout L = qwm::cache_layout(*cfg);
  const int64_t nbh = int64_t(cfg->batch) * cfg->heads, tiles = L.slots / 64;
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<uint32_t> over(static_cast<size_t>(nbh));
  std::vector<uint8_t> ent(static_cast<size_t>(nbh) * 16, 0);
  const uint8_t* c = static_cast<const uint8_t*>(cache);
  hipError_t e = hipMemcpyAsync(over.data(), c + L.k_over, over.size() * 4, hipMemcpyDeviceToHost, s);
  // the directory entry of the tile holding slot n_cache - 1, for every head
  const int64_t T = n_cache > 0 ? (n_cache - 1) / 64 : 0;
  if (e == hipSuccess && n_cache > 0)
    e = hipMemcpy2DAsync(ent.data(), 16, c + L.k_dir + T * 16, size_t(tiles) * 16, 16, size_t(nbh),
                         hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "pool usage readback");
  int64_t used = 0, dropped = 0;
  const int u = int(n_cache - 64 * T);
  const uint64_t below = u >= 64 ? ~uint64_t(0) : ((uint64_t(1) << u) - 1);
  for (int64_t bh = 0; bh < nbh; ++bh) {
    dropped += over[size_t(bh)];
    if (n_cache == 0) continue;
    const uint8_t* p = ent.data() + bh * 16;
    uint32_t base, lo, hi;
    std::memcpy(&base, p, 4);
    std::memcpy(&lo, p + 8, 4);
    std::memcpy(&hi, p + 12, 4);
    used += int64_t(base) + __builtin_popcountll((uint64_t(hi) << 32 | lo) & below);
  }
  *rows_used = used;
  *rows_dropped = dropped;
  return ok();
}

quantwm_status quantwm_logits(const quantwm_config* cfg, const void* calib, const void* cache, int64_t n_cache,
                              const void* q, int64_t n_q, int64_t q_start, int64_t q_first, int32_t frame_tokens,
                              float* logits_out, void* stream) {
  if (!logits_out && n_q > 0) return fail(QWM_ERR_INVALID_ARG, "logits_out is null");
  if (q_first < 0 || q_first > kMaxPositions - (n_q > 0 ? n_q : 0))
    return fail(QWM_ERR_INVALID_ARG, "need 0 <= q_first and q_first + n_q <= %lld", (long long)kMaxPositions);
  return attend_common(cfg, calib, 1, nullptr, cache, n_cache, nullptr, nullptr, 0, q, n_q, q_start, frame_tokens,
                       nullptr, nullptr, logits_out, nullptr, 0, stream, 0, q_first);
}

}  // extern "C"
