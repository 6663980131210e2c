// Quantize-on-append for BF16 Keys and Values on gfx950: QSAC centroid choice
// (Sec. 4.1, Eq. 9-12), group-wise INT2 residual (Eq. 1-4, App. D.1) and PSAC
// coefficients (Sec. 4.2, Eq. 13 and 16) for Keys; nearest centroid + INT2
// residual for Values. The outputs are those of the fp32 kernel; the two
// centroid searches run on the matrix cores.
//
// Mapping: a wave takes 32 consecutive tokens of one (b, h), four waves per
// workgroup. Lanes i and i + 32 share token i and split its channels: lane half
// hf owns channels [hf d/2, (hf + 1) d/2).
//
// Searches. Both are dense products of a (Kc x d) table with the wave's (d x 32)
// tokens,
//     d'_j(t) = b_j + sum_c a_jc x_c(t),
// the expanded Eq. 9 distance (a_jc = -2 w_c mu_jc, b_j = sum_c w_c mu_jc^2) minus
// the centroid-independent sum_c w_c x_c^2, one v_mfma_f32_32x32x16_bf16 per 32
// centroids and 16 channels. The instruction's k index 8 hf + i of step s maps
// to channel hf d/2 + 8 s + i on both operands, so the B operand is the lane's
// own half-row: the token rows load once, straight into operand registers. The
// Key constants a_jc are fp32; the calibration block holds them as three BF16
// planes with an exact sum, so every product is exact in fp32 and only the
// accumulation rounds. The Value table is BF16 and the Value distance uses
// w = 1: the accumulator starts at -b_j / 2, sums mu_jc v_c, and d' is -2 times
// the result, the value the -2 v_c products would give (powers of two scale
// every rounding exactly).
//
// Selection. Each lane keeps the M smallest (d', id) of its candidates in a
// sorted list (ids arrive in increasing order within a lane); the pair merges
// its two lists, both lanes ending with the same M candidates.
//
// Residual and PSAC. Each lane quantises its half-row. Group ranges of a group
// that spans both halves, the 8-bit scales' shared maximum and the Eq. 12 sum
// over groups (added in group order) are combined across the pair with
// v_permlane32_swap. The PSAC projection E U_r runs on the matrix cores as
// well: the errors of each 8-channel residual chunk are the B operand of one k
// step, and one exchange puts the coefficients in rank order on both lanes.
// Everything that turns a float into an integer follows the equations'
// operation order in fp32 with IEEE division and round-to-nearest-even, as in
// the fp32 kernel.
#include "append_common.h"
#include "xcd_order.h"

namespace qwm {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaveTokens = 32, kBlockWaves = 4, kBlockTokens = kWaveTokens * kBlockWaves;

// centroid row (within the 32-row block) of accumulator slot i in lane half hf;
// the lane's column (token) is lane % 32
__device__ inline constexpr int acc_row(int i, int hf) { return (i / 4) * 8 + hf * 4 + (i % 4); }

// the value x holds in lane i ^ 32
__device__ inline uint32_t partner_u32(uint32_t x, int hf) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return hf ? r[0] : r[1];
}
__device__ inline float partner(float x, int hf) { return __uint_as_float(partner_u32(__float_as_uint(x), hf)); }
__device__ inline int partner(int x, int hf) { return int(partner_u32(uint32_t(x), hf)); }

__device__ inline bf16x8 as_frag(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// element E (0..7) of eight BF16 values held as one uint4 (memory order)
__device__ inline float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
template <int E>
__device__ inline float bf_el(const uint4& u) {
  constexpr int k = E / 2;
  const uint32_t w = k == 0 ? u.x : (k == 1 ? u.y : (k == 2 ? u.z : u.w));
  return (E & 1) ? bf_hi(w) : bf_lo(w);
}

// Insert (d, j) into a list sorted by d; j exceeds every id in the list, so an
// equal distance goes after its equals. med3(l[p - 1], d, l[p]) is the new l[p].
template <int MM>
__device__ inline void top_insert(float (&bd)[MM], int (&bi)[MM], float d, int j) {
  bool lt[MM];
#pragma unroll
  for (int p = 0; p < MM; ++p) lt[p] = d < bd[p];
#pragma unroll
  for (int p = MM - 1; p >= 1; --p) {
    const int jp = lt[p] ? j : bi[p];
    bi[p] = lt[p - 1] ? bi[p - 1] : jp;
    bd[p] = __builtin_amdgcn_fmed3f(bd[p - 1], d, bd[p]);
  }
  bi[0] = lt[0] ? j : bi[0];
  bd[0] = lt[0] ? d : bd[0];
}

// Insert (d, j) into a list sorted by (d, id) with any id order.
template <int MM>
__device__ inline void top_insert_lex(float (&bd)[MM], int (&bi)[MM], float d, int j) {
#pragma unroll
  for (int p = 0; p < MM; ++p) {
    const bool lt = (d < bd[p]) | ((d == bd[p]) & (j < bi[p]));
    const float td = lt ? bd[p] : d;
    const int tj = lt ? bi[p] : j;
    bd[p] = lt ? d : bd[p];
    bi[p] = lt ? j : bi[p];
    d = td;
    j = tj;
  }
}

// Pair-merge of the two lanes' top-MM lists: both lanes end with the MM
// smallest (d, id) of the union (ids of the two halves are distinct).
template <int MM>
__device__ inline void merge_pair(float (&bd)[MM], int (&bi)[MM], int hf) {
  float pd[MM];
  int pi[MM];
#pragma unroll
  for (int p = 0; p < MM; ++p) {
    pd[p] = partner(bd[p], hf);
    pi[p] = partner(bi[p], hf);
  }
#pragma unroll
  for (int p = 0; p < MM; ++p) top_insert_lex<MM>(bd, bi, pd[p], pi[p]);
}

// One lane's share of the group structure: DH channels, GL groups of GC
// channels each (a group larger than the half-row spans both lanes: GL = 1).
template <int D, int G>
struct Halves {
  static constexpr int DH = D / 2, NG = D / G;
  static constexpr bool SPAN = G > DH;
  static constexpr int GL = SPAN ? 1 : DH / G, GC = SPAN ? DH : G;
  static __device__ inline int group(int hf, int gl) { return SPAN ? 0 : hf * GL + gl; }
};

// Makes the compiler forget what the packed words hold, so that values unpacked
// from them earlier are not kept live to be reused later (a whole unpacked
// half-row). Emits no instruction.
template <int N>
__device__ inline void forget(uint4 (&u)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(u[i].x), "+v"(u[i].y), "+v"(u[i].z), "+v"(u[i].w));
}

// Residual of the lane's BF16 half-row xh against the half-row mrow of centroid
// z (Eq. 1-2 with q_min = 0, q_max = 3, the range extended to contain 0, the
// residual quantised with the stored scale). Fills the code words of the half
// (16 channels per word), the zero-points, scales (SI8: 8-bit codes and the
// secondary scale) of the lane's groups, and calls each(k, e) with
// e = x_c - (mu_c + s (q_c - z)) for channel c = c0 + k of every 8-channel
// chunk of the half (Eq. 4, Eq. 13), then chunk(c0). The centroid row is read
// from memory 8 channels at a time in each pass (a cached table row); each
// group's range pass precedes its code pass, and with 8-bit scales every range
// pass comes first (the groups share the secondary scale).
template <int D, int G, bool SI8, typename F, typename FC>
__device__ inline void residual_half(uint4 (&xh)[D / 16], const uint4* __restrict__ mrow, int hf,
                                     uint32_t (&cw)[D / 32], int (&zg)[Halves<D, G>::GL],
                                     float (&sg)[Halves<D, G>::GL], int (&cg)[Halves<D, G>::GL], float& sig,
                                     F each, FC chunk) {
  using H = Halves<D, G>;
  constexpr int GL = H::GL, GC = H::GC;
  forget(xh);
  float glo[GL];
  auto range = [&](auto gi, float& lo, float& hi) {
    constexpr int gl = decltype(gi)::value;
    lo = 0.0f;
    hi = 0.0f;
    static_for<0, GC, 8>([&](auto ci) {
      constexpr int c0 = gl * GC + decltype(ci)::value;
      const uint4 mu = mrow[c0 / 8];
      static_for<0, 8>([&](auto ki) {
        constexpr int k = decltype(ki)::value;
        const float r = bf_el<k>(xh[c0 / 8]) - bf_el<k>(mu);
        lo = fminf(lo, r);
        hi = fmaxf(hi, r);
      });
    });
    if constexpr (H::SPAN) {
      lo = fminf(lo, partner(lo, hf));
      hi = fmaxf(hi, partner(hi, hf));
    }
  };
  auto codes = [&](auto gi) {
    constexpr int gl = decltype(gi)::value;
    // unpack the token words and re-read the centroid words here rather than keep
    // the range pass's unpacked values live
    forget(xh);
    asm volatile("" ::: "memory");
    const float s = sg[gl];
    const float sd = s != 0.0f ? s : 1.0f;
    const int z = s != 0.0f ? (int)fminf(fmaxf(rintf(0.0f - glo[gl] / sd), 0.0f), 3.0f) : 0;
    const float inv = s != 0.0f ? 1.0f / s : 0.0f;
    zg[gl] = z;
    static_for<0, GC, 8>([&](auto ci) {
      constexpr int c0 = gl * GC + decltype(ci)::value;
      float xv[8], mu[8], t[8];
      const uint4 m0 = mrow[c0 / 8];
      static_for<0, 8>([&](auto ki) {
        constexpr int k = decltype(ki)::value;
        xv[k] = bf_el<k>(xh[c0 / 8]);
        mu[k] = bf_el<k>(m0);
      });
      round_quotients<8>(xv, mu, s, inv, t);
      uint32_t w = 0;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int q = s != 0.0f ? (int)fminf(fmaxf(t[k] + (float)z, 0.0f), 3.0f) : 0;  // Eq. 1
        w |= uint32_t(q) << (2 * k);
        each(k, xv[k] - (mu[k] + s * (float)(q - z)));
      }
      if constexpr (c0 % 16 == 0) cw[c0 / 16] = w;
      else cw[c0 / 16] |= w << 16;
      chunk(c0);
    });
  };
  if constexpr (SI8) {
    float tg[GL], mx = 0.0f;
    static_for<0, GL>([&](auto gi) {
      constexpr int gl = decltype(gi)::value;
      float lo, hi;
      range(gi, lo, hi);
      glo[gl] = lo;
      tg[gl] = (hi - lo) / 3.0f;
      mx = fmaxf(mx, tg[gl]);
    });
    if constexpr (!H::SPAN) mx = fmaxf(mx, partner(mx, hf));
    sig = f16_round(mx / 255.0f);
#pragma unroll
    for (int gl = 0; gl < GL; ++gl) {
      const int c = sig != 0.0f ? (int)fminf(fmaxf(rintf(tg[gl] / sig), 0.0f), 255.0f) : 0;
      cg[gl] = c;
      sg[gl] = sig * (float)c;  // exact: 11-bit times 8-bit significands
    }
    static_for<0, GL>([&](auto gi) {
      __builtin_amdgcn_sched_barrier(0);
      codes(gi);
    });
  } else {
    static_for<0, GL>([&](auto gi) {
      constexpr int gl = decltype(gi)::value;
      __builtin_amdgcn_sched_barrier(0);
      float lo, hi;
      range(gi, lo, hi);
      glo[gl] = lo;
      sg[gl] = f16_round((hi - lo) / 3.0f);
      codes(gi);
    });
  }
}

// Stores of one token's packed fields for the lane's half: code words, and the
// lane's groups' scales; lane half 0 adds the id, the zero-point bytes (all
// groups) and the SI8 secondary scale.
template <int D, int G, bool SI8>
__device__ inline void store_half(const CacheLayout& L, uint8_t* __restrict__ cache, int64_t codes_sec,
                                  int64_t ids_sec, int64_t zp_sec, int64_t scale_sec, int64_t sigma_sec,
                                  int64_t slot, int hf, bool active, int id, const uint32_t (&cw)[D / 32],
                                  const int (&zg)[Halves<D, G>::GL], const float (&sg)[Halves<D, G>::GL],
                                  const int (&cg)[Halves<D, G>::GL], float sig) {
  using H = Halves<D, G>;
  constexpr int GL = H::GL, NG = H::NG;
  uint32_t zw = 0;
#pragma unroll
  for (int gl = 0; gl < GL; ++gl) zw |= uint32_t(zg[gl]) << (2 * H::group(hf, gl));
  if constexpr (!H::SPAN) zw |= partner_u32(zw, hf);
  if (!active) return;
  uint8_t* cp = cache + codes_sec + slot * (D / 4) + hf * (D / 8);
  if constexpr (D == 128) *reinterpret_cast<uint4*>(cp) = make_uint4(cw[0], cw[1], cw[2], cw[3]);
  else *reinterpret_cast<uint2*>(cp) = make_uint2(cw[0], cw[1]);
  if (hf == 0) {
    cache[ids_sec + slot] = uint8_t(id);
    uint8_t* zp = cache + zp_sec + slot * L.zpb;
    if constexpr (NG > 4) *reinterpret_cast<uint16_t*>(zp) = uint16_t(zw);
    else zp[0] = uint8_t(zw);
    if constexpr (SI8) *reinterpret_cast<uint16_t*>(cache + sigma_sec + slot * 2) = f16_bits(sig);
  }
  if constexpr (H::SPAN) {
    if (hf == 0) {
      if constexpr (SI8) cache[scale_sec + slot] = uint8_t(cg[0]);
      else *reinterpret_cast<uint16_t*>(cache + scale_sec + slot * 2) = f16_bits(sg[0]);
    }
  } else if constexpr (SI8) {
    uint32_t v = 0;
#pragma unroll
    for (int gl = 0; gl < GL; ++gl) v |= uint32_t(cg[gl]) << (8 * gl);
    uint8_t* p = cache + scale_sec + slot * NG + hf * GL;
    if constexpr (GL == 4) *reinterpret_cast<uint32_t*>(p) = v;
    else if constexpr (GL == 2) *reinterpret_cast<uint16_t*>(p) = uint16_t(v);
    else p[0] = uint8_t(v);
  } else {
    uint8_t* p = cache + scale_sec + slot * (2 * NG) + hf * (2 * GL);
    if constexpr (GL == 4) {
      *reinterpret_cast<uint2*>(p) = make_uint2(uint32_t(f16_bits(sg[0])) | uint32_t(f16_bits(sg[1])) << 16,
                                                uint32_t(f16_bits(sg[2])) | uint32_t(f16_bits(sg[3])) << 16);
    } else if constexpr (GL == 2) {
      *reinterpret_cast<uint32_t*>(p) = uint32_t(f16_bits(sg[0])) | uint32_t(f16_bits(sg[1])) << 16;
    } else {
      *reinterpret_cast<uint16_t*>(p) = f16_bits(sg[0]);
    }
  }
}

template <int D, int G, int RP, int MM, bool SI8>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void append_bf16_kernel(const AppendArgs a) {
  using H = Halves<D, G>;
  constexpr int DH = H::DH, NS = D / 16, GL = H::GL;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, n = lane & 31, hf = lane >> 5;
  const int64_t ntb = (a.n_new + kBlockTokens - 1) / kBlockTokens;
  const uint32_t task = qwm_xcd_task(blockIdx.x, gridDim.x);
  const int64_t tb = task % ntb, bh = task / ntb;
  const int64_t b = bh / a.heads, h = bh % a.heads;
  const uint8_t* slab = a.calib + bh * a.slab;

  const int64_t t0 = tb * kBlockTokens + wv * kWaveTokens;
  if (t0 >= a.n_new) return;  // the whole wave is past the chunk
  const int64_t t = t0 + n;
  const bool active = t < a.n_new;
  const int64_t tt = active ? t : a.n_new - 1;  // idle lanes recompute a real token and store nothing
  const int64_t src = ((b * a.n_new + tt) * a.heads + h) * D + hf * DH;
  const int64_t slot = bh * a.L.slots + a.n_cached + tt;
  const int Kc = a.n_centroids, nb = (Kc + 31) / 32;
  const int64_t KD = int64_t(Kc) * D;

  // ---- QSAC candidate search (Eq. 9 expanded) on the matrix cores, top-M by (d', id)
  uint4 xk[NS];
  {
    const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const bf16*>(a.k) + src);
#pragma unroll
    for (int s = 0; s < NS; ++s) xk[s] = p[s];
  }
  float bd[MM];
  int bi[MM];
  // ids start at 0, a valid row: with an infinite or NaN distance (inputs out of
  // range) nothing enters the list, and the score below still reads real rows
#pragma unroll
  for (int p = 0; p < MM; ++p) { bd[p] = __builtin_inff(); bi[p] = 0; }
  {
    const float* __restrict__ bk = reinterpret_cast<const float*>(slab + a.o_b_k);
    const bf16* __restrict__ planes = reinterpret_cast<const bf16*>(slab + a.o_a_k3);
    for (int jb = 0; jb < nb; ++jb) {
      const int j0 = jb * 32;
      f32x16 acc;
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = bk[min(j0 + acc_row(i, hf), Kc - 1)];
      const uint4* arow = reinterpret_cast<const uint4*>(planes + int64_t(min(j0 + n, Kc - 1)) * D + hf * DH);
      // five steps' fragments in flight: steps s + 1 .. s + 4 load while step s multiplies
      constexpr int PF = 5;
      uint4 af[PF][3];
      static_for<0, (PF - 1 < NS ? PF - 1 : NS)>([&](auto pi) {
        constexpr int st = decltype(pi)::value;
#pragma unroll
        for (int pl = 0; pl < 3; ++pl) af[st][pl] = arow[pl * (KD / 8) + st];
      });
      static_for<0, NS>([&](auto si) {
        constexpr int st = decltype(si)::value;
        if constexpr (st + PF - 1 < NS) {
#pragma unroll
          for (int pl = 0; pl < 3; ++pl) af[(st + PF - 1) % PF][pl] = arow[pl * (KD / 8) + st + PF - 1];
        }
#pragma unroll
        for (int pl = 0; pl < 3; ++pl)
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_frag(af[st % PF][pl]), as_frag(xk[st]), acc, 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      });
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int j = j0 + acc_row(i, hf);
        top_insert<MM>(bd, bi, j < Kc ? acc[i] : __builtin_inff(), j);
      }
    }
  }
  merge_pair<MM>(bd, bi, hf);

  // ---- QSAC score (Eq. 10, 12) over the M candidates; ties to the lower id
  const bf16* __restrict__ muk = reinterpret_cast<const bf16*>(slab + a.o_mu_k);
  const float* __restrict__ wg = reinterpret_cast<const float*>(slab + a.o_wg);
  const int M = a.top_m < Kc ? a.top_m : Kc;
  int z = 0;
  float zs = __builtin_inff();
  static_for<0, MM>([&](auto mi) {
    constexpr int m = decltype(mi)::value;
    if (m >= M) return;
    // one candidate row in flight at a time: hoisting all M of them spills
    __builtin_amdgcn_sched_barrier(0);
    const int j = bi[m];
    const uint4* mrow = reinterpret_cast<const uint4*>(muk + int64_t(j) * D + hf * DH);
    float tg[GL];
    static_for<0, GL>([&](auto gi) {
      constexpr int gl = decltype(gi)::value;
      float mx = -__builtin_inff(), mn = __builtin_inff();
      static_for<0, H::GC / 8>([&](auto wi) {
        constexpr int c0 = gl * H::GC + 8 * decltype(wi)::value;
        const uint4 mu = mrow[c0 / 8];
        static_for<0, 8>([&](auto ki) {
          constexpr int k = decltype(ki)::value;
          const float r = bf_el<k>(xk[c0 / 8]) - bf_el<k>(mu);
          mx = fmaxf(mx, r);
          mn = fminf(mn, r);
        });
      });
      if constexpr (H::SPAN) {
        mx = fmaxf(mx, partner(mx, hf));
        mn = fminf(mn, partner(mn, hf));
      }
      const float R = mx - mn;
      tg[gl] = wg[H::group(hf, gl)] * (R * R);
    });
    float S = 0.0f;
    if constexpr (H::SPAN) {
      S = S + tg[0];
    } else {
      float pt[GL];
#pragma unroll
      for (int gl = 0; gl < GL; ++gl) pt[gl] = partner(tg[gl], hf);
#pragma unroll
      for (int gl = 0; gl < GL; ++gl) S = S + (hf ? pt[gl] : tg[gl]);
#pragma unroll
      for (int gl = 0; gl < GL; ++gl) S = S + (hf ? tg[gl] : pt[gl]);
    }
    const bool better = (S < zs) | ((S == zs) & (j < z));
    zs = better ? S : zs;
    z = better ? j : z;
  });

  // ---- Keys: INT2 residual against mu_z, and PSAC (Eq. 13, 16): C = E U_r with
  // E_c = k_c - khat_0,c, on the matrix cores. Each residual chunk is the lane's
  // 8 channels of one k step, so its errors are the B operand as they are made:
  // split into three BF16 parts with an exact sum (as the Key search constants)
  // against the BF16 rows of U_r^T (rank m = lane % 32; zero rows past r), every
  // product is exact and the fp32 accumulator holds ranks acc_row(i, hf).
  // INT8 rows with one FP16 scale (App. D.1).
  {
    const uint4* mrow = reinterpret_cast<const uint4*>(muk + int64_t(z) * D + hf * DH);
    const bf16* __restrict__ ut = reinterpret_cast<const bf16*>(slab + a.o_u_t);
    const int r = a.rank;
    const uint4* urow = reinterpret_cast<const uint4*>(ut + int64_t(min(n, r > 0 ? r - 1 : 0)) * D + hf * DH);
    const bool urank = n < r;
    f32x16 cacc;
#pragma unroll
    for (int i = 0; i < 16; ++i) cacc[i] = 0.0f;
    float ech[8];
    uint32_t cw[D / 32];
    int zg[GL], cg[GL];
    float sg[GL], sig = 0.0f;
    residual_half<D, G, SI8>(
        xk, mrow, hf, cw, zg, sg, cg, sig,
        [&](int k, float e) {
          if constexpr (RP > 0) ech[k] = e;
        },
        [&](int c0) {
          if constexpr (RP > 0) {
            uint4 uf = urow[c0 / 8];
            if (!urank) uf = make_uint4(0u, 0u, 0u, 0u);
            uint32_t p0[4], p1[4], p2[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              uint32_t w0[2], w1[2], w2[2];
#pragma unroll
              for (int u = 0; u < 2; ++u) {
                const float e = ech[2 * q + u];
                w0[u] = __float_as_uint(e) & 0xffff0000u;
                const float r1 = e - __uint_as_float(w0[u]);
                w1[u] = __float_as_uint(r1) & 0xffff0000u;
                w2[u] = __float_as_uint(r1 - __uint_as_float(w1[u])) & 0xffff0000u;
              }
              p0[q] = w0[1] | (w0[0] >> 16);
              p1[q] = w1[1] | (w1[0] >> 16);
              p2[q] = w2[1] | (w2[0] >> 16);
            }
            cacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_frag(uf), as_frag(make_uint4(p0[0], p0[1], p0[2], p0[3])),
                                                           cacc, 0, 0, 0);
            cacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_frag(uf), as_frag(make_uint4(p1[0], p1[1], p1[2], p1[3])),
                                                           cacc, 0, 0, 0);
            cacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_frag(uf), as_frag(make_uint4(p2[0], p2[1], p2[2], p2[3])),
                                                           cacc, 0, 0, 0);
          }
        });
    store_half<D, G, SI8>(a.L, a.cache, a.L.k_codes, a.L.k_ids, a.L.k_zp, a.L.k_scale, a.L.k_sigma, slot, hf,
                          active, z, cw, zg, sg, cg, sig);
    if constexpr (RP > 0) {
      // C in rank order on both lanes: rank k sits in slot (k / 8) * 4 + k % 4 of
      // lane half (k / 4) % 2
      float pc[RP / 2], C[RP];
#pragma unroll
      for (int i = 0; i < RP / 2; ++i) pc[i] = partner(cacc[i], hf);
#pragma unroll
      for (int k = 0; k < RP; ++k) {
        const int i = (k / 8) * 4 + k % 4;
        C[k] = ((k / 4) % 2 == hf) ? cacc[i] : pc[i];
      }
      float amax = 0.0f;
#pragma unroll
      for (int k = 0; k < RP; ++k)
        if (k < r) amax = fmaxf(amax, fabsf(C[k]));
      const float s = f16_round(amax / 127.0f);
      const float sd = s != 0.0f ? s : 1.0f;
      int qc[RP];
#pragma unroll
      for (int k = 0; k < RP; ++k)
        qc[k] = k < r && s != 0.0f ? (int)fminf(fmaxf(rintf(C[k] / sd), -127.0f), 127.0f) : 0;
      // App. D.1 retention: keep the row only if it lowers the lam-weighted
      // error on the principal subspace (ranks in order, fp32)
      bool keep = true;
      if (a.gate) {
        const float* __restrict__ lam = reinterpret_cast<const float*>(slab + a.o_lam);
        float before = 0.0f, after = 0.0f;
#pragma unroll
        for (int k = 0; k < RP; ++k) {
          if (k < r) {
            const float e = C[k] - (float)qc[k] * s;
            before = before + lam[k] * (C[k] * C[k]);
            after = after + lam[k] * (e * e);
          }
        }
        keep = after < before;
      }
      if (active) {
        // with sparse rows the chunk's rows go to the staging rows (row tt of the
        // head) and the commit kernel stores them into the pool
        const int64_t crow = a.L.sparse ? bh * a.L.stage + tt : slot;
        uint8_t* code = a.cache + (a.L.sparse ? a.L.k_st_codes : a.L.k_coef) + crow * r;
        if (r == RP) {
          // the lane's half of the row: RP / 2 bytes
          uint32_t wds[RP / 8];
#pragma unroll
          for (int q = 0; q < RP / 8; ++q) {
            uint32_t v = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int c = hf ? qc[RP / 2 + 4 * q + k] : qc[4 * q + k];
              v |= uint32_t(uint8_t(int8_t(keep ? c : 0))) << (8 * k);
            }
            wds[q] = v;
          }
          if constexpr (RP == 32) *reinterpret_cast<uint4*>(code + 16 * hf) = make_uint4(wds[0], wds[1], wds[2], wds[3]);
          else *reinterpret_cast<uint2*>(code + 8 * hf) = make_uint2(wds[0], wds[1]);
        } else if (hf == 0) {
#pragma unroll
          for (int k = 0; k < RP; ++k)
            if (k < r) code[k] = uint8_t(int8_t(keep ? qc[k] : 0));
        }
        if (hf == 0) {
          *reinterpret_cast<uint16_t*>(a.cache + (a.L.sparse ? a.L.k_st_scale : a.L.k_cscale) + crow * 2) =
              f16_bits(keep ? s : 0.0f);
          if (a.coef_out) {
            float* co = a.coef_out + (bh * a.n_new + tt) * r;
#pragma unroll
            for (int k = 0; k < RP; ++k)
              if (k < r) co[k] = C[k];
          }
        }
      }
    }
  }

  // ---- Values: nearest centroid (w = 1) on the matrix cores, then the same
  // residual path as Keys, no PSAC. (The barrier keeps the Value loads out of
  // the Key residual, where they would only add to its registers.)
  __builtin_amdgcn_sched_barrier(0);
  {
    uint4 xv[NS];
    const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const bf16*>(a.v) + src);
#pragma unroll
    for (int s = 0; s < NS; ++s) xv[s] = p[s];
    const float* __restrict__ bv = reinterpret_cast<const float*>(slab + a.o_b_v);
    const bf16* __restrict__ muv = reinterpret_cast<const bf16*>(slab + a.o_mu_v);
    float dv = __builtin_inff();
    int zv = 0;
    for (int jb = 0; jb < nb; ++jb) {
      const int j0 = jb * 32;
      f32x16 acc;
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = -0.5f * bv[min(j0 + acc_row(i, hf), Kc - 1)];
      const uint4* arow = reinterpret_cast<const uint4*>(muv + int64_t(min(j0 + n, Kc - 1)) * D + hf * DH);
      // the block's fragments all load at once (one per step)
      uint4 af[NS];
#pragma unroll
      for (int st = 0; st < NS; ++st) af[st] = arow[st];
#pragma unroll
      for (int st = 0; st < NS; ++st)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_frag(af[st]), as_frag(xv[st]), acc, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int j = j0 + acc_row(i, hf);
        const float d = -2.0f * acc[i];
        const bool better = (j < Kc) & (d < dv);  // ids increase: ties keep the lower one
        dv = better ? d : dv;
        zv = better ? j : zv;
      }
    }
    {
      const float pd = partner(dv, hf);
      const int pz = partner(zv, hf);
      const bool take = (pd < dv) | ((pd == dv) & (pz < zv));
      dv = take ? pd : dv;
      zv = take ? pz : zv;
    }
    const uint4* mrow = reinterpret_cast<const uint4*>(muv + int64_t(zv) * D + hf * DH);
    uint32_t cw[D / 32];
    int zg[GL], cg[GL];
    float sg[GL], sig = 0.0f;
    residual_half<D, G, SI8>(xv, mrow, hf, cw, zg, sg, cg, sig, [](int, float) {}, [](int) {});
    store_half<D, G, SI8>(a.L, a.cache, a.L.v_codes, a.L.v_ids, a.L.v_zp, a.L.v_scale, a.L.v_sigma, slot, hf,
                          active, zv, cw, zg, sg, cg, sig);
  }
}

template <int D, int G, bool SI8>
hipError_t launch_dgs(const AppendArgs& a, int batch, hipStream_t s) {
  const int64_t ntb = (a.n_new + kBlockTokens - 1) / kBlockTokens;
  const dim3 grid((unsigned)(ntb * a.heads * batch));
  const int rp = a.rank == 0 ? 0 : (a.rank <= 16 ? 16 : 32);  // the [d][rs] stride of U_r
  const bool wide = a.top_m > 4;
  if (rp == 32) {
    if (wide) hipLaunchKernelGGL((append_bf16_kernel<D, G, 32, 8, SI8>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((append_bf16_kernel<D, G, 32, 4, SI8>), grid, dim3(256), 0, s, a);
  } else if (rp == 16) {
    if (wide) hipLaunchKernelGGL((append_bf16_kernel<D, G, 16, 8, SI8>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((append_bf16_kernel<D, G, 16, 4, SI8>), grid, dim3(256), 0, s, a);
  } else {
    if (wide) hipLaunchKernelGGL((append_bf16_kernel<D, G, 0, 8, SI8>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((append_bf16_kernel<D, G, 0, 4, SI8>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

// This file is compiled once per (head_dim, group size): QWM_APPEND_D and
// QWM_APPEND_G select the instantiations.
template <int D, int G>
hipError_t launch_append_bf16(const AppendArgs& a, int batch, hipStream_t s) {
  return a.L.i8 ? launch_dgs<D, G, true>(a, batch, s) : launch_dgs<D, G, false>(a, batch, s);
}

template hipError_t launch_append_bf16<QWM_APPEND_D, QWM_APPEND_G>(const AppendArgs&, int, hipStream_t);

}  // namespace qwm
