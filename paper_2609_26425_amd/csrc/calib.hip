// Calibration kernels for gfx950: the calibration block (centroids, channel
// sensitivities, principal basis) and the constants the append search derives
// from it; the historical Query second moment (Eq. 6) in fp64; and
// deterministic Lloyd K-means for the centroids (Eq. 3).
#include "qwm_common.h"

namespace qwm {
namespace {

__device__ inline float ldf(const float* p) { return *p; }
__device__ inline float ldf(const bf16* p) { return (float)*p; }

// double -> bf16 with one rounding (nearest, ties to even), for normal values.
__device__ inline bf16 to_bf16_rn(double x) {
  uint64_t u = __double_as_longlong(x);
  const uint64_t lsb = (u >> 45) & 1;
  u += (uint64_t(1) << 44) - 1 + lsb;
  u &= ~((uint64_t(1) << 45) - 1);
  return bf16((float)__longlong_as_double(u));  // exact: the value already fits bf16
}
__device__ inline void store_rn(float* p, double x) { *p = (float)x; }
__device__ inline void store_rn(bf16* p, double x) { *p = to_bf16_rn(x); }

// Eq. 12 group sums W_g, the expanded-distance constants of Eq. 9
// (a_jc = -2 (w_c mu_jc), b_j = sum_c (w_c mu_jc) mu_jc; Values use w = 1) and
// U_r in [d][r] order for the append kernel's per-channel PSAC accumulation.
// With the full metric the Key constants expand (k - mu_j)^T Mn (k - mu_j)
// instead: p_j = Mn mu_j (fp32, columns in order), a_jc = -2 p_jc and
// b_j = sum_c p_jc mu_jc; the k^T Mn k term is the same for every centroid.
template <typename T>
__global__ __launch_bounds__(256) void derive_kernel(uint8_t* calib, quantwm_calib_layout C, int d, int G,
                                                     int Kc, int r, int full) {
  uint8_t* slab = calib + int64_t(blockIdx.x) * C.slab_bytes;
  const float* w = reinterpret_cast<const float*>(slab + C.w);
  float* wg = reinterpret_cast<float*>(slab + C.wg);
  const T* mk = reinterpret_cast<const T*>(slab + C.mu_k);
  const T* mv = reinterpret_cast<const T*>(slab + C.mu_v);
  float* ak = reinterpret_cast<float*>(slab + C.a_k);
  float* bk = reinterpret_cast<float*>(slab + C.b_k);
  float* av = reinterpret_cast<float*>(slab + C.a_v);
  float* bv = reinterpret_cast<float*>(slab + C.b_v);
  for (int g = threadIdx.x; g < d / G; g += 256) {
    float s = 0.0f;
    for (int c = g * G; c < (g + 1) * G; ++c) s = s + w[c];
    wg[g] = s;
  }
  const float* mm = reinterpret_cast<const float*>(slab + C.m);
  for (int i = threadIdx.x; i < Kc * d; i += 256) {
    const int c = i % d;
    const float mkv = ldf(mk + i), mvv = ldf(mv + i);
    if (full) {
      const T* mj = mk + (i / d) * d;
      float p = 0.0f;
      for (int c2 = 0; c2 < d; ++c2) p = __builtin_fmaf(mm[c * d + c2], ldf(mj + c2), p);
      ak[i] = -2.0f * p;
    } else {
      ak[i] = -2.0f * (w[c] * mkv);
    }
    av[i] = -2.0f * mvv;
  }
  __syncthreads();  // b_k reads the a_k rows written by other threads
  if constexpr (sizeof(T) == 2) {
    // a_k as three BF16 planes with an exact sum, for the matrix-core search:
    // p0 keeps a's top 8 significant bits (truncated), p1 the top 8 of the exact
    // remainder a - p0, and p2 = a - p0 - p1, which has at most 8 significant
    // bits left and so is a BF16 value (for |a| above 2^-110 or so)
    uint16_t* pl = reinterpret_cast<uint16_t*>(slab + C.a_k3);
    for (int i = threadIdx.x; i < Kc * d; i += 256) {
      const float av0 = ak[i];
      const uint32_t u0 = __float_as_uint(av0) & 0xffff0000u;
      const float r1 = av0 - __uint_as_float(u0);
      const uint32_t u1 = __float_as_uint(r1) & 0xffff0000u;
      const float r2 = r1 - __uint_as_float(u1);
      pl[i] = uint16_t(u0 >> 16);
      pl[Kc * d + i] = uint16_t(u1 >> 16);
      pl[2 * Kc * d + i] = __builtin_bit_cast(uint16_t, bf16(r2));
    }
  }
  const T* ut = reinterpret_cast<const T*>(slab + C.u_t);
  float* udr = reinterpret_cast<float*>(slab + C.u_dr);
  const int rs = r == 0 ? 0 : (r <= 16 ? 16 : 32);
  for (int i = threadIdx.x; i < rs * d; i += 256) {
    const int c = i / rs, k = i % rs;
    udr[i] = k < r ? ldf(ut + k * d + c) : 0.0f;
  }
  for (int j = threadIdx.x; j < Kc; j += 256) {
    float sk = 0.0f, sv = 0.0f;
    for (int c = 0; c < d; ++c) {
      const float mkv = ldf(mk + j * d + c), mvv = ldf(mv + j * d + c);
      // full metric: -0.5 a_jc is p_jc exactly
      sk = __builtin_fmaf(full ? -0.5f * ak[j * d + c] : w[c] * mkv, mkv, sk);
      sv = __builtin_fmaf(mvv, mvv, sv);
    }
    bk[j] = sk;
    bv[j] = sv;
  }
  if constexpr (sizeof(T) == 2) {
    // binary16 copies of the BF16 tables for the attention producers, scaled by a
    // power of two: the table's largest magnitude lands in [2^14, 2^15), so each
    // component of at least 2^-31 of it is exact in binary16 (BF16 keeps 8
    // significant bits) and none overflows
    __shared__ float s_max[2][256];
    float mxk = 0.0f, mxv = 0.0f;
    for (int i = threadIdx.x; i < Kc * d; i += 256) {
      mxk = fmaxf(mxk, fabsf(ldf(mk + i)));
      mxv = fmaxf(mxv, fabsf(ldf(mv + i)));
    }
    s_max[0][threadIdx.x] = mxk;
    s_max[1][threadIdx.x] = mxv;
    __syncthreads();
    for (int st = 128; st > 0; st /= 2) {
      if (threadIdx.x < st) {
        s_max[0][threadIdx.x] = fmaxf(s_max[0][threadIdx.x], s_max[0][threadIdx.x + st]);
        s_max[1][threadIdx.x] = fmaxf(s_max[1][threadIdx.x], s_max[1][threadIdx.x + st]);
      }
      __syncthreads();
    }
    int ek = 0, ev = 0;
    if (s_max[0][0] > 0.0f) { int x; frexpf(s_max[0][0], &x); ek = x - 15; }  // max in [2^(x-1), 2^x)
    if (s_max[1][0] > 0.0f) { int x; frexpf(s_max[1][0], &x); ev = x - 15; }
    _Float16* hk = reinterpret_cast<_Float16*>(slab + C.mu_k16);
    _Float16* hv = reinterpret_cast<_Float16*>(slab + C.mu_v16);
    for (int i = threadIdx.x; i < Kc * d; i += 256) {
      hk[i] = (_Float16)ldexpf(ldf(mk + i), -ek);
      hv[i] = (_Float16)ldexpf(ldf(mv + i), -ev);
    }
    if (threadIdx.x == 0) {
      int32_t* e16 = reinterpret_cast<int32_t*>(slab + C.e16);
      e16[0] = ek;
      e16[1] = ev;
    }
  }
}

// Copy method-level tables into the slabs: mu [BH][Kc][d], w [BH][d],
// u_t [BH][r][d] (zeros if null), lam [BH][r] (zeros if null), and the full
// metric's matrix m [BH][d][d] when given.
template <typename T>
__global__ __launch_bounds__(256) void pack_kernel(uint8_t* calib, quantwm_calib_layout C, int d, int Kc, int r,
                                                   const T* mu_k, const T* mu_v, const float* w, const T* u_t,
                                                   const float* lam, const float* m) {
  const int64_t bh = blockIdx.x;
  uint8_t* slab = calib + bh * C.slab_bytes;
  T* mk = reinterpret_cast<T*>(slab + C.mu_k);
  T* mv = reinterpret_cast<T*>(slab + C.mu_v);
  T* ut = reinterpret_cast<T*>(slab + C.u_t);
  float* wo = reinterpret_cast<float*>(slab + C.w);
  float* lo = reinterpret_cast<float*>(slab + C.lam);
  for (int i = threadIdx.x; i < Kc * d; i += 256) {
    mk[i] = mu_k[bh * Kc * d + i];
    mv[i] = mu_v[bh * Kc * d + i];
  }
  for (int i = threadIdx.x; i < d; i += 256) wo[i] = w[bh * d + i];
  for (int i = threadIdx.x; i < r * d; i += 256) ut[i] = u_t ? u_t[bh * r * d + i] : T(0.0f);
  for (int i = threadIdx.x; i < r; i += 256) lo[i] = lam ? lam[bh * r + i] : 0.0f;
  if (m) {
    float* mo = reinterpret_cast<float*>(slab + C.m);
    for (int i = threadIdx.x; i < d * d; i += 256) mo[i] = m[bh * d * d + i];
  }
}

// Eq. 6 without the 1/N: thread (i, j) sums q_i q_j over the tokens in order,
// in fp64 (each fp32 x fp32 product is exact in fp64), then divides by n.
template <typename T>
__global__ __launch_bounds__(256) void moment_kernel(const T* q, int64_t n, int heads, int d, double* m) {
  const int64_t bh = blockIdx.y;
  const int b = int(bh / heads), h = int(bh % heads);
  const int p = blockIdx.x * 256 + threadIdx.x;
  if (p >= d * d) return;
  const int i = p / d, j = p % d;
  const T* base = q + (int64_t(b) * n * heads + h) * d;
  double acc = 0.0;
  for (int64_t t = 0; t < n; ++t) {
    const T* row = base + t * heads * d;
    acc = __builtin_fma((double)ldf(row + i), (double)ldf(row + j), acc);
  }
  m[bh * d * d + p] = acc / (double)n;
}

// Eq. 6 online: continues the fp64 token-order sums of q q^T from their stored
// values, so a sequence of updates equals one pass over all the tokens.
template <typename T>
__global__ __launch_bounds__(256) void moment_accumulate_kernel(const T* q, int64_t n, int heads, int d, double* sums,
                                                                int64_t* count) {
  const int64_t bh = blockIdx.y;
  const int b = int(bh / heads), h = int(bh % heads);
  const int p = blockIdx.x * 256 + threadIdx.x;
  if (bh == 0 && p == 0) *count += n;
  if (p >= d * d) return;
  const int i = p / d, j = p % d;
  const T* base = q + (int64_t(b) * n * heads + h) * d;
  double acc = sums[bh * d * d + p];
  for (int64_t t = 0; t < n; ++t) {
    const T* row = base + t * heads * d;
    acc = __builtin_fma((double)ldf(row + i), (double)ldf(row + j), acc);
  }
  sums[bh * d * d + p] = acc;
}

template <typename T>
__global__ __launch_bounds__(256) void km_init_kernel(const T* x, int64_t n, int heads, int d, int Kc,
                                                      uint8_t* calib, int64_t slab_bytes, int64_t o_mu) {
  const int64_t bh = blockIdx.x;
  const int b = int(bh / heads), h = int(bh % heads);
  T* mu = reinterpret_cast<T*>(calib + bh * slab_bytes + o_mu);
  for (int i = threadIdx.x; i < Kc * d; i += 256) {
    const int j = i / d, c = i % d;
    const int64_t t = (int64_t(j) * n) / Kc;
    mu[i] = x[((int64_t(b) * n + t) * heads + h) * d + c];
  }
}

// Lloyd assignment: nearest centroid by squared Euclidean distance summed in
// channel order (fp32, no contraction), ties to the lower id.
template <typename T, int D>
__global__ __launch_bounds__(256) void km_assign_kernel(const T* x, int64_t n, int heads, int Kc,
                                                        const uint8_t* calib, int64_t slab_bytes, int64_t o_mu,
                                                        int32_t* assign) {
  const int64_t bh = blockIdx.y;
  const int b = int(bh / heads), h = int(bh % heads);
  const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (t >= n) return;
  const T* __restrict__ mu = reinterpret_cast<const T*>(calib + bh * slab_bytes + o_mu);
  const T* row = x + ((int64_t(b) * n + t) * heads + h) * D;
  float xv[D];
#pragma unroll
  for (int c = 0; c < D; ++c) xv[c] = ldf(row + c);
  int best = 0;
  float bd = 0.0f;
  for (int j = 0; j < Kc; ++j) {
    float acc = 0.0f;
#pragma unroll
    for (int c = 0; c < D; ++c) {
      const float e = xv[c] - ldf(mu + j * D + c);
      acc = acc + e * e;
    }
    if (j == 0 || acc < bd) { best = j; bd = acc; }
  }
  assign[bh * n + t] = best;
}

// Lloyd update: thread (j, c) sums x_tc over the tokens of cluster j in token
// order (fp64), then stores the mean rounded once to the table type; an empty
// cluster keeps its centroid.
template <typename T>
__global__ __launch_bounds__(256) void km_update_kernel(const T* x, int64_t n, int heads, int d, int Kc,
                                                        uint8_t* calib, int64_t slab_bytes, int64_t o_mu,
                                                        const int32_t* assign) {
  const int64_t bh = blockIdx.y;
  const int b = int(bh / heads), h = int(bh % heads);
  const int p = blockIdx.x * 256 + threadIdx.x;
  if (p >= Kc * d) return;
  const int j = p / d, c = p % d;
  const int32_t* as = assign + bh * n;
  const T* base = x + (int64_t(b) * n * heads + h) * d + c;
  double sum = 0.0;
  int64_t cnt = 0;
  for (int64_t t = 0; t < n; ++t)
    if (as[t] == j) {
      sum += (double)ldf(base + t * heads * d);
      ++cnt;
    }
  if (cnt > 0) store_rn(reinterpret_cast<T*>(calib + bh * slab_bytes + o_mu) + p, sum / (double)cnt);
}

template <typename T>
hipError_t kmeans_t(const quantwm_config& c, const T* x, int64_t n, int iters, uint8_t* calib, int64_t o_mu,
                    int32_t* assign, hipStream_t s) {
  const quantwm_calib_layout C = calib_layout(c);
  const int bh = c.batch * c.heads, d = c.head_dim, Kc = c.n_centroids;
  hipLaunchKernelGGL(km_init_kernel<T>, dim3(bh), dim3(256), 0, s, x, n, c.heads, d, Kc, calib, C.slab_bytes, o_mu);
  for (int it = 0; it < iters; ++it) {
    const dim3 ga((unsigned)((n + 255) / 256), (unsigned)bh);
    if (d == 64)
      hipLaunchKernelGGL((km_assign_kernel<T, 64>), ga, dim3(256), 0, s, x, n, c.heads, Kc, calib, C.slab_bytes, o_mu,
                         assign);
    else
      hipLaunchKernelGGL((km_assign_kernel<T, 128>), ga, dim3(256), 0, s, x, n, c.heads, Kc, calib, C.slab_bytes,
                         o_mu, assign);
    const dim3 gu((unsigned)((Kc * d + 255) / 256), (unsigned)bh);
    hipLaunchKernelGGL(km_update_kernel<T>, gu, dim3(256), 0, s, x, n, c.heads, d, Kc, calib, C.slab_bytes, o_mu,
                       assign);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_derive_constants(const quantwm_config& c, uint8_t* calib, hipStream_t s) {
  const quantwm_calib_layout C = calib_layout(c);
  const dim3 grid((unsigned)(c.batch * c.heads));
  const int full = c.metric == QWM_METRIC_FULL;
  if (c.dtype == QWM_BF16)
    hipLaunchKernelGGL(derive_kernel<bf16>, grid, dim3(256), 0, s, calib, C, c.head_dim, c.group_size, c.n_centroids,
                       c.rank, full);
  else
    hipLaunchKernelGGL(derive_kernel<float>, grid, dim3(256), 0, s, calib, C, c.head_dim, c.group_size, c.n_centroids,
                       c.rank, full);
  return hipGetLastError();
}

hipError_t launch_pack_tables(const quantwm_config& c, const void* mu_k, const void* mu_v, const float* w,
                              const void* u_t, const float* lam, const float* m, uint8_t* calib, hipStream_t s) {
  const quantwm_calib_layout C = calib_layout(c);
  const dim3 grid((unsigned)(c.batch * c.heads));
  if (c.dtype == QWM_BF16)
    hipLaunchKernelGGL(pack_kernel<bf16>, grid, dim3(256), 0, s, calib, C, c.head_dim, c.n_centroids, c.rank,
                       (const bf16*)mu_k, (const bf16*)mu_v, w, (const bf16*)u_t, lam, m);
  else
    hipLaunchKernelGGL(pack_kernel<float>, grid, dim3(256), 0, s, calib, C, c.head_dim, c.n_centroids, c.rank,
                       (const float*)mu_k, (const float*)mu_v, w, (const float*)u_t, lam, m);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_derive_constants(c, calib, s);
}

hipError_t launch_second_moment(const quantwm_config& c, const void* q, int64_t n, double* m, hipStream_t s) {
  const int d = c.head_dim;
  const dim3 grid((unsigned)((d * d + 255) / 256), (unsigned)(c.batch * c.heads));
  if (c.dtype == QWM_BF16)
    hipLaunchKernelGGL(moment_kernel<bf16>, grid, dim3(256), 0, s, (const bf16*)q, n, c.heads, d, m);
  else
    hipLaunchKernelGGL(moment_kernel<float>, grid, dim3(256), 0, s, (const float*)q, n, c.heads, d, m);
  return hipGetLastError();
}

hipError_t launch_moment_accumulate(const quantwm_config& c, const void* q, int64_t n, double* sums, int64_t* count,
                                    hipStream_t s) {
  const int d = c.head_dim;
  const dim3 grid((unsigned)((d * d + 255) / 256), (unsigned)(c.batch * c.heads));
  if (c.dtype == QWM_BF16)
    hipLaunchKernelGGL(moment_accumulate_kernel<bf16>, grid, dim3(256), 0, s, (const bf16*)q, n, c.heads, d, sums,
                       count);
  else
    hipLaunchKernelGGL(moment_accumulate_kernel<float>, grid, dim3(256), 0, s, (const float*)q, n, c.heads, d, sums,
                       count);
  return hipGetLastError();
}

hipError_t launch_kmeans(const quantwm_config& c, const void* x, int64_t n, int iters, uint8_t* calib, int64_t o_mu,
                         int32_t* assign, hipStream_t s) {
  if (c.dtype == QWM_BF16) return kmeans_t<bf16>(c, (const bf16*)x, n, iters, calib, o_mu, assign, s);
  return kmeans_t<float>(c, (const float*)x, n, iters, calib, o_mu, assign, s);
}

}  // namespace qwm
