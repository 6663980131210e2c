// Quantize-on-append for fp32 Keys and Values on gfx950: QSAC centroid choice
// (Sec. 4.1, Eq. 9-12), group-wise INT2 residual (Eq. 1-4, App. D.1) and PSAC
// coefficients (Sec. 4.2, Eq. 13 and 16) for Keys; nearest centroid + INT2
// residual for Values. (BF16 Keys and Values: append_bf16.hip, the same outputs
// with the searches on the matrix cores.)
//
// Mapping: one token-head per lane, 256 tokens of one (b, h) per workgroup. The
// candidate search is the dominant cost (Kc * d multiply-adds per token for K
// and again for V). It uses the expanded distance
//     d'_j = b_j + sum_c a_jc k_c,  a_jc = -2 w_c mu_jc,  b_j = sum_c w_c mu_jc^2,
// which equals Eq. 9 minus the centroid-independent sum_c w_c k_c^2, so it has
// the same ordering in exact arithmetic at one FMA per term. a and b are
// wave-uniform and arrive through scalar loads, so the vector ALU does nothing
// but FMAs in the inner loop. Everything that turns a float into an integer
// (the Eq. 12 score, the INT2 and INT8 codes) follows the equations' operation
// order in fp32 with IEEE division and round-to-nearest-even.
#include "append_common.h"

namespace qwm {
namespace {

template <typename T, int D>
__device__ inline void load_row(const T* __restrict__ src, float (&x)[D]) {
  static_assert(sizeof(T) == 4, "fp32 rows");
  const float4* p = reinterpret_cast<const float4*>(src);
#pragma unroll
  for (int i = 0; i < D / 4; ++i) {
    float4 u = p[i];
    x[4 * i] = u.x; x[4 * i + 1] = u.y; x[4 * i + 2] = u.z; x[4 * i + 3] = u.w;
  }
}

// Residual of one token against centroid row mu_row, group by group (Eq. 1-2
// with q_min = 0, q_max = 3, the range extended to contain 0, the residual
// quantised with the stored scale). Token and centroid values stream from
// memory 16 channels at a time in two passes (range, then codes). Codes are
// stored as they are made; `each(c, e)` receives e = x_c - (mu_c + s (q_c - z))
// for every channel c in order (Eq. 4, Eq. 13), and `chunk(c0)` follows the
// last channel of every chunk of CH channels starting at c0.
// SI8 (App. D.1 8-bit group scales): the range passes of all groups come first,
// since the groups share the secondary scale sig = RN16(max_g t_g / 255); a
// group's step is then sig * c_g with c_g = RN(t_g / sig) in [0, 255].
template <typename T, int D, int G, bool SI8, typename F, typename FC>
__device__ inline void quant_stream(const T* __restrict__ xrow, const T* __restrict__ mrow,
                                    uint8_t* __restrict__ codes, bool active, int (&zg)[D / G],
                                    float (&sg)[D / G], int (&cg)[D / G], float& sig, F each, FC chunk) {
  constexpr int CH = G < 16 ? G : 16;
  constexpr int NG = D / G;
  // 0-extended residual range of group g
  auto range = [&](auto gi, float& lo, float& hi) {
    constexpr int g = decltype(gi)::value;
    lo = 0.0f;
    hi = 0.0f;
    static_for<0, G, CH>([&](auto ci) {
      constexpr int c0 = g * G + decltype(ci)::value;
      float xv[CH], mu[CH];
      load_row<T, CH>(xrow + c0, xv);
      load_row<T, CH>(mrow + c0, mu);
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const float r = xv[c] - mu[c];
        lo = r < lo ? r : lo;
        hi = r > hi ? r : hi;
      }
    });
  };
  float glo[SI8 ? NG : 1];
  if constexpr (SI8) {
    float tg[NG], mx = 0.0f;
    static_for<0, NG>([&](auto gi) {
      constexpr int g = decltype(gi)::value;
      __builtin_amdgcn_sched_barrier(0);
      float lo, hi;
      range(gi, lo, hi);
      glo[g] = lo;
      tg[g] = (hi - lo) / 3.0f;
      mx = tg[g] > mx ? tg[g] : mx;
    });
    sig = f16_round(mx / 255.0f);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int c = sig != 0.0f ? (int)fminf(fmaxf(rintf(tg[g] / sig), 0.0f), 255.0f) : 0;
      cg[g] = c;
      sg[g] = sig * (float)c;  // exact: 11-bit times 8-bit significands
    }
  }
  static_for<0, NG>([&](auto gi) {
    constexpr int g = decltype(gi)::value;
    // keep each group's loads inside the group: hoisting them all ahead would
    // hold every chunk in registers at once
    __builtin_amdgcn_sched_barrier(0);
    float lo;
    if constexpr (SI8) {
      lo = glo[g];
    } else {
      float hi;
      range(gi, lo, hi);
      sg[g] = f16_round((hi - lo) / 3.0f);
    }
    const float s = sg[g];
    const float sd = s != 0.0f ? s : 1.0f;
    const int z = s != 0.0f ? (int)fminf(fmaxf(rintf(0.0f - lo / sd), 0.0f), 3.0f) : 0;
    const float inv = s != 0.0f ? 1.0f / s : 0.0f;
    zg[g] = z;
    static_for<0, G, CH>([&](auto ci) {
      constexpr int c0 = g * G + decltype(ci)::value;
      float xv[CH], mu[CH];
      load_row<T, CH>(xrow + c0, xv);
      load_row<T, CH>(mrow + c0, mu);
      float t[CH];
      round_quotients<CH>(xv, mu, s, inv, t);
      uint32_t cw = 0;
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const int q = s != 0.0f ? (int)fminf(fmaxf(t[c] + (float)z, 0.0f), 3.0f) : 0;  // Eq. 1
        cw |= uint32_t(q) << (2 * c);
        each(c0 + c, xv[c] - (mu[c] + s * (float)(q - z)));
      }
      if (active) {
        if constexpr (CH == 16) *reinterpret_cast<uint32_t*>(codes + c0 / 4) = cw;
        else *reinterpret_cast<uint16_t*>(codes + c0 / 4) = uint16_t(cw);
      }
      chunk(c0);
    });
  });
}

// zero-points (INT2, four per byte) and the group scales: binary16 steps, or
// (SI8) the 8-bit codes c_g and the binary16 secondary scale
template <int D, int G, bool SI8>
__device__ inline void store_meta(uint8_t* __restrict__ zp_dst, uint8_t* __restrict__ scale_dst,
                                  uint8_t* __restrict__ sigma_dst, const int (&zg)[D / G],
                                  const float (&sg)[D / G], const int (&cg)[D / G], float sig) {
  constexpr int NG = D / G;
  uint32_t z = 0;
#pragma unroll
  for (int g = 0; g < NG; ++g) z |= uint32_t(zg[g]) << (2 * g);
  zp_dst[0] = uint8_t(z & 255);
  if constexpr (NG > 4) zp_dst[1] = uint8_t(z >> 8);
  if constexpr (SI8) {
#pragma unroll
    for (int g = 0; g < NG; ++g) scale_dst[g] = uint8_t(cg[g]);
    *reinterpret_cast<uint16_t*>(sigma_dst) = f16_bits(sig);
  } else {
    uint16_t* sp = reinterpret_cast<uint16_t*>(scale_dst);
#pragma unroll
    for (int g = 0; g < NG; ++g) sp[g] = f16_bits(sg[g]);
  }
}

// Bubble (dist, id) into a list kept sorted by (dist, id); ids arrive in
// increasing order, so a strict comparison keeps the lower id first on ties.
template <int MM>
__device__ inline void topm_insert(float (&bd)[MM], int (&bi)[MM], float dv, int iv) {
#pragma unroll
  for (int p = 0; p < MM; ++p) {
    const bool lt = dv < bd[p];
    const float td = lt ? bd[p] : dv;
    const int ti = lt ? bi[p] : iv;
    bd[p] = lt ? dv : bd[p];
    bi[p] = lt ? iv : bi[p];
    dv = td;
    iv = ti;
  }
}

template <typename T, int D, int G, int RP, int MM, bool SI8>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void append_kernel(const AppendArgs a) {
  constexpr int NG = D / G;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const bool active = t < a.n_new;
  const int64_t tt = active ? t : a.n_new - 1;  // idle lanes recompute a real token and store nothing
  const int64_t bh = int64_t(b) * a.heads + h;
  const uint8_t* slab = a.calib + bh * a.slab;
  const float* __restrict__ ak = reinterpret_cast<const float*>(slab + a.o_a_k);
  const float* __restrict__ bk = reinterpret_cast<const float*>(slab + a.o_b_k);
  const float* __restrict__ av = reinterpret_cast<const float*>(slab + a.o_a_v);
  const float* __restrict__ bv = reinterpret_cast<const float*>(slab + a.o_b_v);
  const float* __restrict__ wg = reinterpret_cast<const float*>(slab + a.o_wg);
  const T* __restrict__ muk = reinterpret_cast<const T*>(slab + a.o_mu_k);
  const T* __restrict__ muv = reinterpret_cast<const T*>(slab + a.o_mu_v);
  const float* __restrict__ udr = reinterpret_cast<const float*>(slab + a.o_u_dr);
  const int Kc = a.n_centroids;
  const int64_t src = ((int64_t(b) * a.n_new + tt) * a.heads + h) * D;
  const int64_t slot = bh * a.L.slots + a.n_cached + tt;

  float x[D];
  load_row<T, D>(reinterpret_cast<const T*>(a.k) + src, x);

  // ---- QSAC candidate search (Eq. 9, expanded form), top-M by (d', id)
  float bd[MM];
  int bi[MM];
  // ids start at 0, a valid row: with an infinite or NaN distance (inputs out of
  // range) nothing enters the list, and the score below still reads real rows
#pragma unroll
  for (int p = 0; p < MM; ++p) { bd[p] = __builtin_inff(); bi[p] = 0; }
  for (int j = 0; j < Kc; j += 4) {
    float acc[4];
    int row[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      row[u] = min(j + u, Kc - 1);
      acc[u] = bk[row[u]];
    }
#pragma unroll
    for (int c = 0; c < D; ++c)
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] = __builtin_fmaf(ak[row[u] * D + c], x[c], acc[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (j + u < Kc) topm_insert<MM>(bd, bi, acc[u], j + u);
  }

  // ---- QSAC score (Eq. 10, 12) over the M candidates; ties to the lower id
  const int M = a.top_m < Kc ? a.top_m : Kc;
  int z = 0;
  float zs = __builtin_inff();
  static_for<0, MM>([&](auto mi) {
    constexpr int m = decltype(mi)::value;
    if (m >= M) return;
    const int j = bi[m];
    const T* mrow = muk + int64_t(j) * D;
    float S = 0.0f;
    static_for<0, NG>([&](auto gi) {
      constexpr int g = decltype(gi)::value;
      float mx = -__builtin_inff(), mn = __builtin_inff();
#pragma unroll
      for (int c0 = 0; c0 < G; c0 += 16) {
        float mu[16];
        load_row<T, 16>(mrow + g * G + c0, mu);
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          const float r = x[g * G + c0 + c] - mu[c];
          mx = r > mx ? r : mx;
          mn = r < mn ? r : mn;
        }
      }
      const float R = mx - mn;
      S = S + wg[g] * (R * R);
    });
    if (S < zs || (S == zs && j < z)) { zs = S; z = j; }
  });

  // ---- Values: nearest centroid (w = 1). Both searches run before the first
  // store, so the compiler may keep their table loads on the scalar path.
  int zv = 0;
  float dv = __builtin_inff();
  // branch-free argmin update: a divergent branch here turns the table loads of
  // the loop into per-lane vector loads
  auto take = [&](int j, const float (&acc)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool better = (j + u < Kc) & (acc[u] < dv);
      dv = better ? acc[u] : dv;
      zv = better ? j + u : zv;
    }
  };
  {
    load_row<T, D>(reinterpret_cast<const T*>(a.v) + src, x);
    for (int j = 0; j < Kc; j += 4) {
      float acc[4];
      int row[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        row[u] = min(j + u, Kc - 1);
        acc[u] = bv[row[u]];
      }
#pragma unroll
      for (int c = 0; c < D; ++c)
#pragma unroll
        for (int u = 0; u < 4; ++u) acc[u] = __builtin_fmaf(av[row[u] * D + c], x[c], acc[u]);
      take(j, acc);
    }
  }
  // ---- INT2 residual against mu_z, with PSAC accumulated channel by channel:
  // E_c = k_c - khat_0,c (Eq. 13), C_k += E_c U_ck (Eq. 16). From here on the
  // key is re-read 16 channels at a time (L1 hits), so only the r accumulators
  // stay resident. INT8 rows with one FP16 scale (App. D.1).
  {
    const T* krow = reinterpret_cast<const T*>(a.k) + src;
    const T* mrow = muk + int64_t(z) * D;
    float C[RP > 0 ? RP : 1];
#pragma unroll
    for (int k = 0; k < (RP > 0 ? RP : 1); ++k) C[k] = 0.0f;
    int zg[NG], cg[NG];
    float sg[NG], sig = 0.0f;
    // The errors of one chunk go to this thread's LDS row, and a rolled loop over
    // the chunk's channels adds e_c U_r[c, :] to C. Written as straight-line code,
    // the compiler hoisted the wave-uniform loads of all d x RP entries of U_r
    // and spilled them.
    constexpr int CHK = G < 16 ? G : 16, ES = CHK + 1;
    __shared__ float s_err[RP > 0 ? 256 * ES : 1];
    float* my_err = s_err + threadIdx.x * ES;
    quant_stream<T, D, G, SI8>(
        krow, mrow, a.cache + a.L.k_codes + slot * (D / 4), active, zg, sg, cg, sig,
        [&](int c, float e) {
          if constexpr (RP > 0) my_err[c % CHK] = e;
        },
        [&](int c0) {
          if constexpr (RP > 0) {
#pragma nounroll
            for (int c = 0; c < CHK; ++c) {
              const float e = my_err[c];
              const float* urow = udr + (c0 + c) * RP;
#pragma unroll
              for (int k = 0; k < RP; ++k) C[k] = __builtin_fmaf(e, urow[k], C[k]);
            }
          }
        });
    if (active) {
      store_meta<D, G, SI8>(a.cache + a.L.k_zp + slot * a.L.zpb, a.cache + a.L.k_scale + slot * a.L.sb,
                            a.cache + a.L.k_sigma + slot * 2, zg, sg, cg, sig);
      a.cache[a.L.k_ids + slot] = uint8_t(z);
    }
    if constexpr (RP > 0) {
      const int r = a.rank;
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
        int8_t* code = reinterpret_cast<int8_t*>(a.cache + (a.L.sparse ? a.L.k_st_codes : a.L.k_coef) + crow * r);
        float* co = a.coef_out ? a.coef_out + (bh * a.n_new + tt) * r : nullptr;
#pragma unroll
        for (int k = 0; k < RP; ++k) {
          if (k < r) {
            code[k] = int8_t(keep ? qc[k] : 0);
            if (co) co[k] = C[k];
          }
        }
        *reinterpret_cast<uint16_t*>(a.cache + (a.L.sparse ? a.L.k_st_scale : a.L.k_cscale) + crow * 2) =
            f16_bits(keep ? s : 0.0f);
      }
    }
  }

  // ---- Values: the same residual path as Keys, no PSAC
  {
    int zg[NG], cg[NG];
    float sg[NG], sig = 0.0f;
    quant_stream<T, D, G, SI8>(reinterpret_cast<const T*>(a.v) + src, muv + int64_t(zv) * D,
                               a.cache + a.L.v_codes + slot * (D / 4), active, zg, sg, cg, sig, [](int, float) {},
                               [](int) {});
    if (active) {
      store_meta<D, G, SI8>(a.cache + a.L.v_zp + slot * a.L.zpb, a.cache + a.L.v_scale + slot * a.L.sb,
                            a.cache + a.L.v_sigma + slot * 2, zg, sg, cg, sig);
      a.cache[a.L.v_ids + slot] = uint8_t(zv);
    }
  }
}

template <typename T, int D, int G, bool SI8>
hipError_t launch_dgs(const AppendArgs& a, int batch, hipStream_t s) {
  const dim3 grid((unsigned)((a.n_new + 255) / 256), (unsigned)a.heads, (unsigned)batch);
  const int rp = a.rank == 0 ? 0 : (a.rank <= 16 ? 16 : 32);  // the [d][rs] stride of U_r
  const bool wide = a.top_m > 4;
  if (rp == 32) {
    if (wide) hipLaunchKernelGGL((append_kernel<T, D, G, 32, 8, SI8>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((append_kernel<T, D, G, 32, 4, SI8>), grid, dim3(256), 0, s, a);
  } else if (rp == 16) {
    if (wide) hipLaunchKernelGGL((append_kernel<T, D, G, 16, 8, SI8>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((append_kernel<T, D, G, 16, 4, SI8>), grid, dim3(256), 0, s, a);
  } else {
    if (wide) hipLaunchKernelGGL((append_kernel<T, D, G, 0, 8, SI8>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((append_kernel<T, D, G, 0, 4, SI8>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

// This file is compiled once per (head_dim, group size): QWM_APPEND_D and
// QWM_APPEND_G select the instantiations.
template <int D, int G>
hipError_t launch_append_f32(const AppendArgs& a, int batch, hipStream_t s) {
  return a.L.i8 ? launch_dgs<float, D, G, true>(a, batch, s) : launch_dgs<float, D, G, false>(a, batch, s);
}

template hipError_t launch_append_f32<QWM_APPEND_D, QWM_APPEND_G>(const AppendArgs&, int, hipStream_t);

}  // namespace qwm
