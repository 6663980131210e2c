// Host side of the attention launches: key-split count, LDS sizes, dispatch
// to the kernel instances (one translation unit per element type, head_dim
// and PSAC rank padding) and the log-sum-exp merge of partial results.
#include "attend_shape.h"

namespace qwm {
namespace {

// Merges the n_split partial results of every Query: with M the largest running
// max and w_s = 2^((m_s - M) log2(e) / sqrt(d)), O = sum w_s O_s / sum w_s l_s
// and lse = M / sqrt(d) + log(sum w_s l_s), the sums taken in split order. One
// wave per Query, D / 64 contiguous channels per lane. The planes are read four
// splits per trip so that their loads are in flight together (a split count
// known only at run time otherwise leaves one split's loads in flight at a time).
template <typename T, int D>
__global__ __launch_bounds__(256) void attend_combine(const AttendArgs a) {
  const int64_t qi = int64_t(blockIdx.x) * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  const int h = blockIdx.y, b = blockIdx.z;
  if (qi >= a.n_q) return;
  const int64_t bh = int64_t(b) * a.heads + h;
  const int64_t plane = int64_t(a.heads) * gridDim.z * a.n_q;  // rows per split
  const float mscale = 1.4426950408889634f / sqrtf((float)D);
  constexpr int PL = D / 64;
  typedef float vecf __attribute__((ext_vector_type(PL)));
  const float2* ml = reinterpret_cast<const float2*>(a.part_ml);
  float M = -__builtin_inff();
  for (int sp = 0; sp < a.n_split; ++sp) M = fmaxf(M, ml[sp * plane + bh * a.n_q + qi].x);
  vecf o = {};
  float L = 0.0f;
  auto add = [&](const float2 p, const vecf v) __attribute__((always_inline)) {
    if (!(p.y > 0.0f)) return;  // this split saw no visible key of this Query
    const float w = __builtin_amdgcn_exp2f((p.x - M) * mscale);
    L += w * p.y;
#pragma unroll
    for (int j = 0; j < PL; ++j) o[j] += w * v[j];
  };
  auto row_of = [&](int sp) { return sp * plane + bh * a.n_q + qi; };
  auto vals = [&](int sp) { return *reinterpret_cast<const vecf*>(a.part_o + row_of(sp) * D + lane * PL); };
  int sp = 0;
  for (; sp + 4 <= a.n_split; sp += 4) {
    float2 p[4];
    vecf v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      p[u] = ml[row_of(sp + u)];
      v[u] = vals(sp + u);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) add(p[u], v[u]);
  }
  for (; sp < a.n_split; ++sp) add(ml[row_of(sp)], vals(sp));
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  T* orow = reinterpret_cast<T*>(a.out) + ((int64_t(b) * a.n_q + qi) * a.heads + h) * D + lane * PL;
#pragma unroll
  for (int j = 0; j < PL; ++j) orow[j] = T(o[j] * inv);
  if (a.lse && lane == 0) a.lse[bh * a.n_q + qi] = L > 0.0f ? M / sqrtf((float)D) + logf(L) : -__builtin_inff();
}

template <typename T, int D>
hipError_t launch_d(const AttendArgs& a, int batch, bool logits, hipStream_t s) {
  hipError_t e;
  if (a.rank == 0) e = launch_attend_rp<T, D, 0>(a, batch, logits, s);
  else if (a.rank <= 16) e = launch_attend_rp<T, D, 16>(a, batch, logits, s);
  else e = launch_attend_rp<T, D, 32>(a, batch, logits, s);
  if (e != hipSuccess || logits || a.n_split == 1 || a.partial) return e;
  hipLaunchKernelGGL((attend_combine<T, D>), dim3((unsigned)((a.n_q + 3) / 4), (unsigned)a.heads, (unsigned)batch),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

size_t attend_lds_bytes(int d, int elem, int rank, int n_centroids, bool tables) {
  if (elem == 2) return d == 64 ? attend_lds_bytes_t<bf16, 64>(rank, n_centroids, tables)
                                : attend_lds_bytes_t<bf16, 128>(rank, n_centroids, tables);
  return d == 64 ? attend_lds_bytes_t<float, 64>(rank, n_centroids, tables)
                 : attend_lds_bytes_t<float, 128>(rank, n_centroids, tables);
}
int attend_splits(int64_t n_q, int heads, int batch, int64_t n_cache, int cus) {
  // Split the key range only when the launch gives fewer than two workgroups
  // per compute unit (one runs per CU). The split count minimises the rounds of
  // workgroups times each one's work: its share of the key tiles plus a fixed
  // cost of about 32 tiles (table staging, Query fragments, pipeline fill,
  // partial write), up to 16 splits of at least 8 tiles.
  const int64_t wgs = (n_q + BQ - 1) / BQ * heads * batch;
  if (wgs <= 0 || wgs >= 2 * int64_t(cus)) return 1;
  const int64_t tiles = (n_cache + KT - 1) / KT;
  int best = 1;
  int64_t best_cost = -1;
  for (int ns = 1; ns <= 16; ++ns) {
    if (ns > 1 && tiles / ns < 8) break;
    const int64_t rounds = (wgs * ns + cus - 1) / cus;
    const int64_t cost = rounds * ((tiles + ns - 1) / ns + 32);
    if (best_cost < 0 || cost < best_cost) {
      best = ns;
      best_cost = cost;
    }
  }
  return best;
}

bool attend_tables_fit(int d, int elem, int rank, int n_centroids) {
  return attend_lds_bytes(d, elem, rank, n_centroids, true) <= kLdsLimit;
}

hipError_t launch_attend_f32(const AttendArgs& a, int d, int batch, bool logits, hipStream_t s) {
  if (d == 64) return launch_d<float, 64>(a, batch, logits, s);
  if (d == 128) return launch_d<float, 128>(a, batch, logits, s);
  return hipErrorInvalidValue;
}

// merges the a.n_split partial planes of a.part_o / a.part_ml into a.out and a.lse
hipError_t launch_attend_combine(const AttendArgs& a, int d, int batch, bool is_bf16, hipStream_t s) {
  const dim3 grid((unsigned)((a.n_q + 3) / 4), (unsigned)a.heads, (unsigned)batch);
  if (is_bf16) {
    if (d == 64) hipLaunchKernelGGL((attend_combine<bf16, 64>), grid, dim3(256), 0, s, a);
    else if (d == 128) hipLaunchKernelGGL((attend_combine<bf16, 128>), grid, dim3(256), 0, s, a);
    else return hipErrorInvalidValue;
  } else {
    if (d == 64) hipLaunchKernelGGL((attend_combine<float, 64>), grid, dim3(256), 0, s, a);
    else if (d == 128) hipLaunchKernelGGL((attend_combine<float, 128>), grid, dim3(256), 0, s, a);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attend_bf16(const AttendArgs& a, int d, int batch, bool logits, hipStream_t s) {
  if (d == 64) return launch_d<bf16, 64>(a, batch, logits, s);
  if (d == 128) return launch_d<bf16, 128>(a, batch, logits, s);
  return hipErrorInvalidValue;
}

}  // namespace qwm
