// Tile geometry of the attention kernel, shared by the kernel instances and
// the host-side launch helpers.
#pragma once

#include "qwm_common.h"

namespace qwm {

// Workgroup: NC consumer waves (32 Queries each: logits, softmax, P.V on the
// matrix cores) and NP producer waves (read and dequantise the packed tiles).
// Waves w and w + 4 share a SIMD, so every SIMD runs one producer beside two
// consumers: the producer's vector work overlaps the consumers' matrix work.
constexpr int NC = 8, NP = 4, BQ = 32 * NC, KT = kAttendTileKeys, NT = 64 * (NC + NP), PT = 64 * NP;

// LDS row strides (elements), chosen so that the matrix-core operand reads are
// free of bank conflicts: K tile rows of 272 B (16-byte reads), V^T rows of
// 136 B and chat rows of (r + 4) * 2 B (8-byte reads), and centroid-table rows
// padded by 16 B so that lanes looking up different centroids spread over banks.
template <typename T, int D, int RP>
struct Lds {
  static constexpr bool H = sizeof(T) == 2;
  static constexpr int KS = D + (H ? 8 : 1);
  static constexpr int CS = (RP > 0 ? RP : 1) + (H ? 4 : 1);
  static constexpr int VS = KT + (H ? 4 : 1);
  static constexpr int TS = D + (H ? 8 : 4);
  static constexpr int tile_elems = KT * KS + KT * CS + D * VS;
};

// LDS bytes of one launch: two tile buffers, plus the centroid tables when staged.
template <typename T, int D>
inline size_t attend_lds_bytes_t(int rank, int kc, bool tables) {
  size_t tile = 0;
  if (rank == 0) tile = Lds<T, D, 0>::tile_elems;
  else if (rank <= 16) tile = Lds<T, D, 16>::tile_elems;
  else tile = Lds<T, D, 32>::tile_elems;
  constexpr size_t TS = Lds<T, D, 0>::TS;
  return (2 * tile + (tables ? size_t(2) * kc * TS : 0)) * sizeof(T);
}

// LDS the kernels may use (MI355X: 160 KB per compute unit).
constexpr size_t kLdsLimit = 160 * 1024;

// Kernel instances for one (element type, head_dim, PSAC rank padding), each
// compiled in a translation unit of its own. The combine kernel is launched by
// the caller.
template <typename T, int D, int RP>
hipError_t launch_attend_rp(const AttendArgs& a, int batch, bool logits, hipStream_t s);

}  // namespace qwm
