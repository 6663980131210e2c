// Per-chunk PSAC coefficient records (App. D.1 storage): the INT8 rows and
// FP16 scales of cache slots [start, start + n) of every (b, h), written as a
// dense record or as a sparse one that keeps only the rows with a non-zero
// scale, whichever is smaller once the sparse indices are counted. The record
// format is documented with quantwm_coef_pack in include/quantwm.h.
#include "qwm_common.h"

namespace qwm {
namespace {

constexpr int kHeader = 16;

__device__ inline uint16_t ld16(const uint8_t* p) { return uint16_t(p[0] | (uint32_t(p[1]) << 8)); }
__device__ inline uint32_t ld32(const uint8_t* p) {
  return uint32_t(p[0]) | (uint32_t(p[1]) << 8) | (uint32_t(p[2]) << 16) | (uint32_t(p[3]) << 24);
}
__device__ inline void st16(uint8_t* p, uint16_t v) {
  p[0] = uint8_t(v);
  p[1] = uint8_t(v >> 8);
}
__device__ inline void st32(uint8_t* p, uint32_t v) {
  for (int i = 0; i < 4; ++i) p[i] = uint8_t(v >> (8 * i));
}

// Byte offset of head bh's block in a sparse record: the header, the counts,
// then (r + 4) bytes per kept row of the heads before it.
__device__ inline int64_t sparse_block(const uint8_t* rec, int64_t nbh, int64_t bh, int r) {
  int64_t off = kHeader + 4 * nbh;
  for (int64_t i = 0; i < bh; ++i) off += int64_t(ld32(rec + kHeader + 4 * i)) * (r + 4);
  return off;
}

// kept rows (non-zero FP16 scale) of head blockIdx.x -> u32 at counts + 4 bh
__global__ __launch_bounds__(256) void coef_count_kernel(const uint8_t* cache, CacheLayout L, int64_t start, int n,
                                                         uint8_t* counts) {
  const int64_t bh = blockIdx.x;
  const uint8_t* sc = cache + L.k_cscale + (bh * L.slots + start) * 2;
  uint32_t c = 0;
  for (int t = threadIdx.x; t < n; t += 256) c += ld16(sc + 2 * t) != 0;
  __shared__ uint32_t tot;
  if (threadIdx.x == 0) tot = 0;
  __syncthreads();
  atomicAdd(&tot, c);
  __syncthreads();
  if (threadIdx.x == 0) st32(counts + 4 * bh, tot);
}

__global__ void coef_header_kernel(uint8_t* rec, uint32_t layout, uint32_t n, uint32_t r, uint32_t nbh) {
  st32(rec, layout);
  st32(rec + 4, n);
  st32(rec + 8, r);
  st32(rec + 12, nbh);
}

// dense: codes [BH][n][r], then scales [BH][n]; one thread per row
template <bool PACK>
__global__ __launch_bounds__(256) void coef_dense_kernel(uint8_t* cache, CacheLayout L, int64_t start, int n,
                                                         uint8_t* rec, int64_t nbh) {
  const int64_t bh = blockIdx.y;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= n) return;
  const int r = L.r;
  const int64_t slot = bh * L.slots + start + t, row = bh * n + t;
  uint8_t* c = cache + L.k_coef + slot * r;
  uint8_t* s = cache + L.k_cscale + slot * 2;
  uint8_t* rc = rec + kHeader + row * r;
  uint8_t* rs = rec + kHeader + nbh * n * r + row * 2;
  for (int i = 0; i < r; ++i) {
    if (PACK) rc[i] = c[i];
    else c[i] = rc[i];
  }
  if (PACK) {
    rs[0] = s[0];
    rs[1] = s[1];
  } else {
    s[0] = rs[0];
    s[1] = rs[1];
  }
}

// sparse pack, one workgroup per head: the kept rows in slot order, each at its
// rank among the kept rows (wave ballots, then the waves' totals in LDS). The
// head's count was written by coef_count_kernel; a row past it is not written.
__global__ __launch_bounds__(256) void coef_sparse_pack_kernel(const uint8_t* cache, CacheLayout L, int64_t start,
                                                               int n, uint8_t* rec, int64_t nbh) {
  const int64_t bh = blockIdx.x;
  const int r = L.r;
  const uint32_t cnt = ld32(rec + kHeader + 4 * bh);
  uint8_t* idx = rec + sparse_block(rec, nbh, bh, r);
  uint8_t* codes = idx + 2 * int64_t(cnt);
  uint8_t* scales = codes + int64_t(r) * cnt;
  const int lane = threadIdx.x % 64, w = threadIdx.x / 64;
  __shared__ uint32_t wsum[4];
  uint32_t base = 0;
  for (int t0 = 0; t0 < n; t0 += 256) {
    const int t = t0 + threadIdx.x;
    const int64_t slot = bh * L.slots + start + t;
    const bool keep = t < n && ld16(cache + L.k_cscale + slot * 2) != 0;
    const uint64_t m = __ballot(keep);
    const uint32_t below = uint32_t(__popcll(m & ((uint64_t(1) << lane) - 1)));
    if (lane == 0) wsum[w] = uint32_t(__popcll(m));
    __syncthreads();
    uint32_t pos = base + below;
    for (int i = 0; i < w; ++i) pos += wsum[i];
    const uint32_t tot = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    if (keep && pos < cnt) {
      st16(idx + 2 * int64_t(pos), uint16_t(t));
      const uint8_t* c = cache + L.k_coef + slot * r;
      for (int i = 0; i < r; ++i) codes[int64_t(pos) * r + i] = c[i];
      scales[2 * int64_t(pos)] = cache[L.k_cscale + slot * 2];
      scales[2 * int64_t(pos) + 1] = cache[L.k_cscale + slot * 2 + 1];
    }
    base += tot;
    __syncthreads();  // wsum is rewritten by the next batch
  }
}

// sparse unpack, one workgroup per head: zero the chunk's rows, then write the
// record's rows at their slots (indices at or past n are skipped)
__global__ __launch_bounds__(256) void coef_sparse_unpack_kernel(uint8_t* cache, CacheLayout L, int64_t start, int n,
                                                                 const uint8_t* rec, int64_t nbh) {
  const int64_t bh = blockIdx.x;
  const int r = L.r;
  for (int t = threadIdx.x; t < n; t += 256) {
    const int64_t slot = bh * L.slots + start + t;
    for (int i = 0; i < r; ++i) cache[L.k_coef + slot * r + i] = 0;
    cache[L.k_cscale + slot * 2] = 0;
    cache[L.k_cscale + slot * 2 + 1] = 0;
  }
  __syncthreads();
  const uint32_t cnt = ld32(rec + kHeader + 4 * bh);
  const uint8_t* idx = rec + sparse_block(rec, nbh, bh, r);
  const uint8_t* codes = idx + 2 * int64_t(cnt);
  const uint8_t* scales = codes + int64_t(r) * cnt;
  for (uint32_t m = threadIdx.x; m < cnt; m += 256) {
    const int t = ld16(idx + 2 * int64_t(m));
    if (t >= n) continue;
    const int64_t slot = bh * L.slots + start + t;
    for (int i = 0; i < r; ++i) cache[L.k_coef + slot * r + i] = codes[int64_t(m) * r + i];
    cache[L.k_cscale + slot * 2] = scales[2 * int64_t(m)];
    cache[L.k_cscale + slot * 2 + 1] = scales[2 * int64_t(m) + 1];
  }
}

}  // namespace

hipError_t launch_coef_count(const quantwm_config& c, const void* cache, int64_t start, int n, void* counts,
                             hipStream_t s) {
  const CacheLayout L = cache_layout(c);
  hipLaunchKernelGGL(coef_count_kernel, dim3(unsigned(c.batch * c.heads)), dim3(256), 0, s,
                     static_cast<const uint8_t*>(cache), L, start, n, static_cast<uint8_t*>(counts));
  return hipGetLastError();
}

hipError_t launch_coef_pack(const quantwm_config& c, const void* cache, int64_t start, int n, void* record,
                            int layout, hipStream_t s) {
  const CacheLayout L = cache_layout(c);
  const int64_t nbh = int64_t(c.batch) * c.heads;
  uint8_t* rec = static_cast<uint8_t*>(record);
  uint8_t* cch = const_cast<uint8_t*>(static_cast<const uint8_t*>(cache));  // read only when packing
  if (layout == QWM_COEF_SPARSE) {
    // the counts the sparse writer reads are already in the record
    hipLaunchKernelGGL(coef_sparse_pack_kernel, dim3(unsigned(nbh)), dim3(256), 0, s, cch, L, start, n, rec, nbh);
  } else if (n > 0) {
    hipLaunchKernelGGL(coef_dense_kernel<true>, dim3(unsigned((n + 255) / 256), unsigned(nbh)), dim3(256), 0, s, cch,
                       L, start, n, rec, nbh);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the header goes in last: a dense record's codes start where the counts were
  hipLaunchKernelGGL(coef_header_kernel, dim3(1), dim3(1), 0, s, rec, uint32_t(layout), uint32_t(n),
                     uint32_t(c.rank), uint32_t(nbh));
  return hipGetLastError();
}

hipError_t launch_coef_unpack(const quantwm_config& c, const void* record, int layout, void* cache, int64_t start,
                              int n, hipStream_t s) {
  const CacheLayout L = cache_layout(c);
  const int64_t nbh = int64_t(c.batch) * c.heads;
  const uint8_t* rec = static_cast<const uint8_t*>(record);
  if (layout == QWM_COEF_SPARSE)
    hipLaunchKernelGGL(coef_sparse_unpack_kernel, dim3(unsigned(nbh)), dim3(256), 0, s, static_cast<uint8_t*>(cache),
                       L, start, n, rec, nbh);
  else if (n > 0)
    hipLaunchKernelGGL(coef_dense_kernel<false>, dim3(unsigned((n + 255) / 256), unsigned(nbh)), dim3(256), 0, s,
                       static_cast<uint8_t*>(cache), L, start, n, const_cast<uint8_t*>(rec), nbh);
  return hipGetLastError();
}


namespace {

// Stores the staged rows of one append call (slots [n_cached, n_cached + n)) of
// head blockIdx.x into its pool: every row (dense) or the rows with a non-zero
// scale (sparse), whichever is smaller with one mask bit per slot as the sparse
// index (ties dense); rows in slot order after the rows of the slots below; a
// row past the pool's end is counted and not stored. Then the directory of the
// chunk's tiles: the tile holding n_cached keeps its rows below n_cached. One
// wave per 64-slot tile, four tiles per pass.
__global__ __launch_bounds__(256) void coef_commit_kernel(uint8_t* cache, CacheLayout L, int64_t n_cached, int n) {
  const int64_t bh = blockIdx.x;
  const int r = L.r, tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int64_t tiles = L.slots / 64;
  uint8_t* dir = cache + L.k_dir + bh * tiles * 16;
  const uint8_t* st_c = cache + L.k_st_codes + bh * L.stage * r;
  const uint8_t* st_s = cache + L.k_st_scale + bh * L.stage * 2;
  uint8_t* pc = cache + L.k_coef + bh * L.pool * r;
  uint8_t* ps = cache + L.k_cscale + bh * L.pool * 2;
  __shared__ uint32_t s_cnt[4];
  __shared__ int64_t s_fill;
  __shared__ uint32_t s_kept;
  // pool rows used by the slots below n_cached (read before this block writes)
  if (tid == 0) {
    int64_t f = 0;
    if (n_cached > 0) {
      const int64_t T = (n_cached - 1) / 64;
      const int used = int(n_cached - 64 * T);
      const uint64_t below = used == 64 ? ~uint64_t(0) : ((uint64_t(1) << used) - 1);
      const uint8_t* e = dir + T * 16;
      const uint64_t m = uint64_t(ld32(e + 8)) | (uint64_t(ld32(e + 12)) << 32);
      f = int64_t(ld32(e)) + __popcll(m & below);
    }
    s_fill = f;
    s_kept = 0;
  }
  __syncthreads();
  uint32_t c = 0;
  for (int t = tid; t < n; t += 256) c += ld16(st_s + 2 * t) != 0;
  atomicAdd(&s_kept, c);
  __syncthreads();
  const int64_t kept = s_kept, fill = s_fill;
  const bool sparse = kept * (r + 2) + (n + 7) / 8 < int64_t(n) * (r + 2);
  const int64_t T0 = n_cached / 64, T1 = (n_cached + n + 63) / 64;  // the chunk's tiles [T0, T1)
  int64_t stored_before = 0;  // stored rows of the chunk before the current pass
  uint32_t over = 0;
  for (int64_t Tp = T0; Tp < T1; Tp += 4) {
    const int64_t T = Tp + wave;
    const int64_t slot = T * 64 + lane, t = slot - n_cached;
    const bool in = T < T1 && t >= 0 && t < n;
    const bool stored = in && (!sparse || ld16(st_s + 2 * t) != 0);
    const uint64_t sb = __ballot(stored);
    const int64_t rank = __popcll(sb & ((uint64_t(1) << lane) - 1));  // stored rows of this tile below the lane
    if (lane == 0) s_cnt[wave] = __popcll(sb);
    __syncthreads();
    int64_t before = stored_before;  // stored rows of the chunk before tile T
    for (int w = 0; w < wave; ++w) before += s_cnt[w];
    const int64_t pass_total = int64_t(s_cnt[0]) + s_cnt[1] + s_cnt[2] + s_cnt[3];
    const int64_t pos = fill + before + rank;
    const bool fit = stored && pos < L.pool;
    if (stored && !fit) ++over;
    if (fit) {
      for (int i = 0; i < r; ++i) pc[pos * r + i] = st_c[t * r + i];
      ps[pos * 2] = st_s[2 * t];
      ps[pos * 2 + 1] = st_s[2 * t + 1];
    }
    const uint64_t fb = __ballot(fit);
    if (lane == 0 && T < T1) {
      uint8_t* e = dir + T * 16;
      uint64_t m = fb;
      if (T * 64 < n_cached) {
        // the chunk starts inside this tile: its rows below n_cached stay
        const int i0 = int(n_cached - T * 64);
        const uint64_t old = uint64_t(ld32(e + 8)) | (uint64_t(ld32(e + 12)) << 32);
        m |= old & ((uint64_t(1) << i0) - 1);
      } else {
        const int64_t b0 = fill + before < L.pool ? fill + before : L.pool;
        st32(e, uint32_t(b0));
        st32(e + 4, 0);
      }
      st32(e + 8, uint32_t(m));
      st32(e + 12, uint32_t(m >> 32));
    }
    stored_before += pass_total;
    __syncthreads();  // s_cnt is reused by the next pass
  }
  // rows without room in the pool, summed over the block
  __shared__ uint32_t s_over;
  if (tid == 0) s_over = 0;
  __syncthreads();
  if (over) atomicAdd(&s_over, over);
  __syncthreads();
  if (tid == 0 && s_over) st32(cache + L.k_over + bh * 4, ld32(cache + L.k_over + bh * 4) + s_over);
}

}  // namespace

hipError_t launch_coef_commit(const quantwm_config& c, void* cache, int64_t n_cached, int64_t n, hipStream_t s) {
  const CacheLayout L = cache_layout(c);
  hipLaunchKernelGGL(coef_commit_kernel, dim3(unsigned(int64_t(c.batch) * c.heads)), dim3(256), 0, s,
                     static_cast<uint8_t*>(cache), L, n_cached, int(n));
  return hipGetLastError();
}

}  // namespace qwm
