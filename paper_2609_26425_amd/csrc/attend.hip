// Chunked attention over the packed 2-bit cache for gfx950 (Eq. 5 with the
// PSAC correction of Eq. 17), Keys and Values dequantised on chip.
//
// Per workgroup: one (b, h) and BQ = 256 Queries (8 waves x 32). The centroid
// tables of the head are staged in LDS once. For every 64-key tile the workgroup
// reads the packed tile (codes, ids, zero-points, scales, INT8 coefficients)
// from HBM, rebuilds
//     khat_0 = mu_z + s (q - z)   (Eq. 4, fp32, then the MFMA type)
//     chat   = code * cscale      (INT8 PSAC row)
//     vhat   = nu_z + s (q - z)
// into LDS (K row-major, V transposed), and every wave then computes its logits
// tile with matrix cores as S^T = [khat_0 | chat] [q | qU_r]^T over an augmented
// depth d + r, so (qU)c is added to qk^T before the softmax. With S^T each lane
// holds one Query column, so the exponentials feed the P.V product straight
// from the accumulator registers and O^T = Vhat^T P^T accumulates in registers.
// Softmax is online (running max and sum per Query, base-2 exponentials).
#include "qwm_common.h"

#include <type_traits>

namespace qwm {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <typename T>
struct Mfma;
template <>
struct Mfma<bf16> {  // v_mfma_f32_32x32x16_bf16
  static constexpr int KPL = 8, KSTEP = 16;
  typedef bf16x8 V;
  static __device__ inline f32x16 run(V a, V b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<float> {  // v_mfma_f32_32x32x2_f32
  static constexpr int KPL = 1, KSTEP = 2;
  typedef float V;
  static __device__ inline f32x16 run(V a, V b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

template <typename V, typename T>
__device__ inline void vset(V& v, int j, T x) {
  if constexpr (sizeof(V) == sizeof(T)) v = x;
  else v[j] = x;
}

// Row of the 32x32 accumulator held by accumulator slot i of a lane in half hf.
__device__ inline constexpr int acc_row(int i, int hf) { return (i / 4) * 8 + hf * 4 + (i % 4); }

template <typename T, int N>
__device__ inline void load_vals(const T* p, float (&out)[N]) {
  if constexpr (sizeof(T) == 2) {
    static_assert(N % 8 == 0 || N == 4, "bf16 loads of 8 or 4 values");
    if constexpr (N == 4) {
      const uint2 u = *reinterpret_cast<const uint2*>(p);
      out[0] = __uint_as_float(u.x << 16); out[1] = __uint_as_float(u.x & 0xffff0000u);
      out[2] = __uint_as_float(u.y << 16); out[3] = __uint_as_float(u.y & 0xffff0000u);
    } else {
#pragma unroll
      for (int i = 0; i < N / 8; ++i) {
        const uint4 u = reinterpret_cast<const uint4*>(p)[i];
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          out[8 * i + 2 * k] = __uint_as_float(w[k] << 16);
          out[8 * i + 2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
        }
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) out[i] = p[i];
  }
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ inline uint32_t pack_bf16(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

template <typename T, int N>
__device__ inline void store_vals(T* p, const float (&x)[N]) {
  if constexpr (sizeof(T) == 2) {
    static_assert(N % 8 == 0, "bf16 stores of 8 values");
#pragma unroll
    for (int i = 0; i < N / 8; ++i)
      reinterpret_cast<uint4*>(p)[i] = make_uint4(pack_bf16(x[8 * i], x[8 * i + 1]), pack_bf16(x[8 * i + 2], x[8 * i + 3]),
                                                  pack_bf16(x[8 * i + 4], x[8 * i + 5]), pack_bf16(x[8 * i + 6], x[8 * i + 7]));
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) p[i] = x[i];
  }
}

// Stores with 8-byte alignment only (rows whose stride is an odd multiple of 8 B).
template <typename T, int N>
__device__ inline void store_vals8(T* p, const float (&x)[N]) {
  if constexpr (sizeof(T) == 2) {
    static_assert(N % 4 == 0, "bf16 stores of 4 values");
#pragma unroll
    for (int i = 0; i < N / 4; ++i)
      reinterpret_cast<uint2*>(p)[i] = make_uint2(pack_bf16(x[4 * i], x[4 * i + 1]), pack_bf16(x[4 * i + 2], x[4 * i + 3]));
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) p[i] = x[i];
  }
}

template <typename T>
__device__ inline void store_pair(T* p, float a, float b) {
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<uint32_t*>(p) = pack_bf16(a, b);
  } else {
    p[0] = a;
    p[1] = b;
  }
}

// INT2 codes of N consecutive channels (channel c in bits 2c of cw) as floats.
// The four 2-bit fields of every byte are spread into four words of bytes, so
// each code converts with one v_cvt_f32_ubyteN.
template <int N>
__device__ inline void codes_to_float(uint32_t cw, float (&q)[N]) {
  const uint32_t w[4] = {cw & 0x03030303u, (cw >> 2) & 0x03030303u, (cw >> 4) & 0x03030303u,
                         (cw >> 6) & 0x03030303u};
#pragma unroll
  for (int c = 0; c < N; ++c) q[c] = (float)((w[c % 4] >> (8 * (c / 4))) & 0xffu);
}

// Builds a bf16x8 MFMA operand from 8 floats with paired conversions.
template <typename V>
__device__ inline V pack_operand(const float* x) {
  if constexpr (sizeof(V) == 16) {
    const uint4 u = make_uint4(pack_bf16(x[0], x[1]), pack_bf16(x[2], x[3]), pack_bf16(x[4], x[5]), pack_bf16(x[6], x[7]));
    return __builtin_bit_cast(V, u);
  } else {
    return x[0];
  }
}

constexpr int NW = 8, BQ = 32 * NW, KT = 64, NT = 64 * NW;

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

template <typename T, int D, int RP, bool LOGITS, bool TAB>
__global__ __launch_bounds__(NT) void attend_kernel(const AttendArgs a) {
  typedef Mfma<T> MF;
  typedef typename MF::V V;
  constexpr int KPL = MF::KPL, KSTEP = MF::KSTEP;
  typedef Lds<T, D, RP> LY;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  T* smem = reinterpret_cast<T*>(smem_raw);
  const int Kc = a.n_centroids;
  // LDS: [mu_K table][mu_V table] (TAB) then two tile buffers, each
  // [K tile][chat tile][V^T tile]. Every LDS pointer is formed as smem + offset
  // where it is used, so the compiler keeps LDS addressing (ds_read/ds_write).
  T* tabK = smem;
  T* tabV = smem + Kc * LY::TS;
  const int tile0 = TAB ? 2 * Kc * LY::TS : 0;

  const int tid = threadIdx.x, wave = tid / 64, lane = tid % 64, l32 = lane % 32, hf = lane / 32;
  const int h = blockIdx.y, b = blockIdx.z;
  const int64_t bh = int64_t(b) * a.heads + h;
  const uint8_t* slab = a.calib + bh * a.slab;
  const T* gtabK = reinterpret_cast<const T*>(slab + a.o_mu_k);
  const T* gtabV = reinterpret_cast<const T*>(slab + a.o_mu_v);
  const T* gU = reinterpret_cast<const T*>(slab + a.o_u_t);
  const CacheLayout& L = a.L;
  const uint8_t* cache = a.cache;
  const int64_t slot0 = bh * L.slots;
  const int r = a.rank;
  const int G = D / L.ng;

  // ---- stage the centroid tables of this head (App. D.1: BF16 centroids)
  if constexpr (TAB) {
    constexpr int PER_ROW = D * int(sizeof(T)) / 16;  // 16-byte chunks per centroid row
    const uint4* sk = reinterpret_cast<const uint4*>(gtabK);
    const uint4* sv = reinterpret_cast<const uint4*>(gtabV);
    for (int i = tid; i < Kc * PER_ROW; i += NT) {
      const int row = i / PER_ROW, ch = i % PER_ROW;
      *reinterpret_cast<uint4*>(tabK + row * LY::TS + ch * (16 / int(sizeof(T)))) = sk[i];
      *reinterpret_cast<uint4*>(tabV + row * LY::TS + ch * (16 / int(sizeof(T)))) = sv[i];
    }
  }

  // ---- Query fragment (B operand: k = channel, column = Query)
  const int64_t qa = int64_t(blockIdx.x) * BQ;
  const int64_t qi = qa + wave * 32 + l32;
  const bool qvalid = qi < a.n_q;
  const T* qrow = reinterpret_cast<const T*>(a.q) + ((int64_t(b) * a.n_q + (qvalid ? qi : 0)) * a.heads + h) * D;
  V qreg[D / KSTEP];
#pragma unroll
  for (int st = 0; st < D / KSTEP; ++st) {
#pragma unroll
    for (int j = 0; j < KPL; ++j) vset(qreg[st], j, qvalid ? qrow[st * KSTEP + hf * KPL + j] : T(0.0f));
  }

  // ---- u = q U_r on matrix cores (A operand: rows = ranks of U_r^T)
  V ureg[RP > 0 ? RP / KSTEP : 1];
  if constexpr (RP > 0) {
    f32x16 uacc;
#pragma unroll
    for (int i = 0; i < 16; ++i) uacc[i] = 0.0f;
#pragma unroll
    for (int st = 0; st < D / KSTEP; ++st) {
      V av;
#pragma unroll
      for (int j = 0; j < KPL; ++j)
        vset(av, j, l32 < r ? gU[int64_t(l32) * D + st * KSTEP + hf * KPL + j] : T(0.0f));
      uacc = MF::run(av, qreg[st], uacc);
    }
    // slot i holds rank acc_row(i, hf): round to the MFMA type (the operand of Eq. 17)
#pragma unroll
    for (int st = 0; st < RP / KSTEP; ++st)
#pragma unroll
      for (int j = 0; j < KPL; ++j) vset(ureg[st], j, T(uacc[st * KPL + j]));
  }

  // ---- key range of this workgroup
  const int64_t F = a.frame_tokens, qs = a.q_start, nc = a.n_cache;
  const int64_t qb = qa + BQ < a.n_q ? qa + BQ : a.n_q;
  int64_t kend = LOGITS ? nc : qs + ((qb - 1) / F + 1) * F;
  if (kend > nc) kend = nc;
  int64_t kfull = qs + (qa / F + 1) * F;  // keys below are visible to every Query of the workgroup
  if (kfull > nc) kfull = nc;
  int64_t lim = qvalid ? qs + (qi / F + 1) * F : nc;  // this lane's Query sees keys j < lim
  if (lim > nc) lim = nc;

  float m_run = -__builtin_inff(), l_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[cb][i] = 0.0f;

  constexpr int CHK = D * KT / NT;        // K channels per thread (one key)
  constexpr int CHV = D * KT / (2 * NT);  // V channels per thread (two keys)
  constexpr int RCH = 8;                  // PSAC ranks per thread
  constexpr int RPT = RP > 0 ? RP / RCH : 1;
  const int kkey = tid / (D / CHK), kch0 = (tid % (D / CHK)) * CHK, kg = kch0 / G;
  const int vkp = tid % (KT / 2), vch0 = (tid / (KT / 2)) * CHV, vg = vch0 / G;
  const int ckey = tid / RPT, cr0 = (tid % RPT) * RCH;
  const bool crole = RP > 0 && tid < KT * RPT && cr0 < r;
  const bool r8 = (r & 7) == 0;

  // ---- packed tile fields of this thread, loaded one tile ahead of use
  uint32_t k_cw = 0, c_lo = 0, c_hi = 0, v_cw[2] = {0, 0};
  int k_id = 0, k_z = 0, v_id[2] = {0, 0}, v_z[2] = {0, 0};
  float k_s = 0.0f, c_s = 0.0f, v_s[2] = {0.0f, 0.0f};
  // per-head field bases (wave-uniform) and 32-bit token offsets inside the head
  const uint8_t* __restrict__ kcb = cache + L.k_codes + slot0 * (D / 4) + kch0 / 4;
  const uint8_t* __restrict__ kib = cache + L.k_ids + slot0;
  const uint8_t* __restrict__ kzb = cache + L.k_zp + slot0 * L.zpb + kg / 4;
  const uint8_t* __restrict__ ksb = cache + L.k_scale + slot0 * 2 * L.ng + 2 * kg;
  const uint8_t* __restrict__ ccb = cache + L.k_coef + slot0 * r + cr0;
  const uint8_t* __restrict__ csb = cache + L.k_cscale + slot0 * 2;
  const uint8_t* __restrict__ vcb = cache + L.v_codes + slot0 * (D / 4) + vch0 / 4;
  const uint8_t* __restrict__ vib = cache + L.v_ids + slot0;
  const uint8_t* __restrict__ vzb = cache + L.v_zp + slot0 * L.zpb + vg / 4;
  const uint8_t* __restrict__ vsb = cache + L.v_scale + slot0 * 2 * L.ng + 2 * vg;
  const uint32_t zpb = L.zpb, sstride = 2 * L.ng, ncu = uint32_t(nc);

  // FULL: every key of the tile is < n_cache, so no per-thread guards. A key
  // past n_cache (tail tiles only) gets centroid 0, scale 0 and code 0: a finite
  // placeholder whose logit the mask turns into -inf, so it never contributes.
  auto load_raw = [&](auto full_tag, uint32_t k0) {
    constexpr bool FULL = decltype(full_tag)::value;
    {
      const uint32_t tok = k0 + kkey;
      if (FULL || tok < ncu) {
        const int id = kib[tok];
        k_id = id < Kc ? id : Kc - 1;
        k_z = (kzb[tok * zpb] >> (2 * (kg % 4))) & 3;
        k_s = (float)*reinterpret_cast<const _Float16*>(ksb + tok * sstride);
        if constexpr (CHK == 16) k_cw = *reinterpret_cast<const uint32_t*>(kcb + tok * (D / 4));
        else k_cw = *reinterpret_cast<const uint16_t*>(kcb + tok * (D / 4));
      } else {
        k_id = 0; k_z = 0; k_s = 0.0f; k_cw = 0;
      }
    }
    if constexpr (RP > 0) {
      const uint32_t tok = k0 + ckey;
      c_s = 0.0f;
      c_lo = 0;
      c_hi = 0;
      if (crole && (FULL || tok < ncu)) {
        c_s = (float)*reinterpret_cast<const _Float16*>(csb + tok * 2);
        const uint8_t* cp = ccb + tok * uint32_t(r);
        if (r8) {
          const uint2 u = *reinterpret_cast<const uint2*>(cp);
          c_lo = u.x;
          c_hi = u.y;
        } else {
          uint32_t w[2] = {0, 0};
#pragma unroll
          for (int k = 0; k < RCH; ++k)
            if (cr0 + k < r) w[k / 4] |= uint32_t(cp[k]) << (8 * (k % 4));
          c_lo = w[0];
          c_hi = w[1];
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const uint32_t tok = k0 + 2 * vkp + e;
      if (FULL || tok < ncu) {
        const int id = vib[tok];
        v_id[e] = id < Kc ? id : Kc - 1;
        v_z[e] = (vzb[tok * zpb] >> (2 * (vg % 4))) & 3;
        v_s[e] = (float)*reinterpret_cast<const _Float16*>(vsb + tok * sstride);
        if constexpr (CHV == 8) v_cw[e] = *reinterpret_cast<const uint16_t*>(vcb + tok * (D / 4));
        else v_cw[e] = vcb[tok * (D / 4)];
      } else {
        v_id[e] = 0; v_z[e] = 0; v_s[e] = 0.0f; v_cw[e] = 0;
      }
    }
  };

  // ---- rebuild khat_0 = mu + s (q - z) (Eq. 4), chat = code * cscale and vhat
  // into tile buffer `buf`. s (q - z) is exact in fp32, so the fma rounds once,
  // exactly like mu + s (q - z).
  auto dequant = [&](int buf) {
    T* kt = smem + tile0 + buf * LY::tile_elems;
    T* ct = kt + KT * LY::KS;
    T* vt = ct + KT * LY::CS;
    {
      float q[CHK], mu[CHK], x[CHK];
      codes_to_float<CHK>(k_cw, q);
      if constexpr (TAB) load_vals<T, CHK>(tabK + k_id * LY::TS + kch0, mu);
      else load_vals<T, CHK>(gtabK + k_id * D + kch0, mu);
      const float zf = (float)k_z;
#pragma unroll
      for (int c = 0; c < CHK; ++c) x[c] = __builtin_fmaf(k_s, q[c] - zf, mu[c]);
      store_vals<T, CHK>(kt + kkey * LY::KS + kch0, x);
    }
    if constexpr (RP > 0) {
      if (tid < KT * RPT) {
        float x[RCH];
#pragma unroll
        for (int k = 0; k < RCH; ++k)
          x[k] = (float)int8_t(((k < 4 ? c_lo : c_hi) >> (8 * (k % 4))) & 255) * c_s;
        store_vals8<T, RCH>(ct + ckey * LY::CS + cr0, x);
      }
    }
    {
      float x0[CHV], x1[CHV];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        float* x = e == 0 ? x0 : x1;
        float q[CHV], mu[CHV];
        codes_to_float<CHV>(v_cw[e], q);
        if constexpr (TAB) load_vals<T, CHV>(tabV + v_id[e] * LY::TS + vch0, mu);
        else load_vals<T, CHV>(gtabV + v_id[e] * D + vch0, mu);
        const float zf = (float)v_z[e];
#pragma unroll
        for (int c = 0; c < CHV; ++c) x[c] = __builtin_fmaf(v_s[e], q[c] - zf, mu[c]);
      }
#pragma unroll
      for (int c = 0; c < CHV; ++c) store_pair<T>(vt + (vch0 + c) * LY::VS + 2 * vkp, x0[c], x1[c]);
    }
  };

  const int64_t ntile = (kend + KT - 1) / KT;
  const int64_t nfull = nc / KT;  // tiles [0, nfull) hold no key past n_cache
  using Full = std::integral_constant<bool, true>;
  using Tail = std::integral_constant<bool, false>;
  if (ntile > 0) {
    if (nfull > 0) load_raw(Full{}, 0u);
    else load_raw(Tail{}, 0u);
    dequant(0);
    if (ntile > 1) {
      if (nfull > 1) load_raw(Full{}, uint32_t(KT));
      else load_raw(Tail{}, uint32_t(KT));
    }
  }
  const float mscale = 1.4426950408889634f / sqrtf((float)D);  // logits are exponentiated as 2^(S log2(e)/sqrt(d))

  for (int64_t it = 0; it < ntile; ++it) {
    const int64_t k0 = it * KT;
    // buffer it&1 is complete and every wave is done with buffer (it+1)&1
    __syncthreads();
    const T* kt = smem + tile0 + int(it & 1) * LY::tile_elems;
    const T* ct = kt + KT * LY::KS;
    const T* vt = ct + KT * LY::CS;

    // ---- logits tile S^T (keys x Queries) on matrix cores
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[kb][i] = 0.0f;
    }
#pragma unroll
    for (int st = 0; st < D / KSTEP; ++st) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const T* krow = kt + (kb * 32 + l32) * LY::KS;
        V av;
        if constexpr (KPL == 8) av = *reinterpret_cast<const V*>(krow + st * KSTEP + hf * KPL);
        else av = krow[st * KSTEP + hf];
        sacc[kb] = MF::run(av, qreg[st], sacc[kb]);
      }
    }
    if constexpr (RP > 0) {
#pragma unroll
      for (int st = 0; st < RP / KSTEP; ++st) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const T* crow = ct + (kb * 32 + l32) * LY::CS;
          V av;
#pragma unroll
          for (int j = 0; j < KPL; ++j) vset(av, j, crow[acc_row(st * KPL + j, hf)]);
          sacc[kb] = MF::run(av, ureg[st], sacc[kb]);
        }
      }
    }

    // ---- next tile into the other buffer while the matrix cores run
    if (it + 1 < ntile) {
      dequant(int((it + 1) & 1));
      if (it + 2 < ntile) {
        if (it + 2 < nfull) load_raw(Full{}, uint32_t(k0 + 2 * KT));
        else load_raw(Tail{}, uint32_t(k0 + 2 * KT));
      }
    }

    if constexpr (LOGITS) {
      if (qvalid) {
        const float inv = 1.0f / sqrtf((float)D);
        float* lrow = a.logits + (bh * a.n_q + qi) * nc;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int64_t j = k0 + kb * 32 + acc_row(i, hf);
            if (j < nc) lrow[j] = j < lim ? sacc[kb][i] * inv : -__builtin_inff();
          }
      }
    } else {
      // ---- online softmax on raw logits; masked keys -> -inf
      if (k0 + KT > kfull) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i)
            if (k0 + kb * 32 + acc_row(i, hf) >= lim) sacc[kb][i] = -__builtin_inff();
      }
      float mt = -__builtin_inff();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) mt = fmaxf(mt, sacc[kb][i]);
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float m_new = fmaxf(m_run, mt);
      if (__any(m_new > m_run)) {  // rescale only when some row's running max moved
        const float alpha = m_new == -__builtin_inff() ? 1.0f : __builtin_amdgcn_exp2f((m_run - m_new) * mscale);
        l_run *= alpha;
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
          for (int i = 0; i < 16; ++i) oacc[cb][i] *= alpha;
        m_run = m_new;
      }
      const float mc = m_run == -__builtin_inff() ? 0.0f : -m_run * mscale;
      float lpart[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][i], mscale, mc));
          sacc[kb][i] = p;
          lpart[i % 4] += p;
        }
      l_run += (lpart[0] + lpart[1]) + (lpart[2] + lpart[3]);

      // ---- O^T += Vhat^T P^T (B operand = this lane's probabilities)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int t = 0; t < 32 / KSTEP; ++t) {
          float pv[KPL];
#pragma unroll
          for (int j = 0; j < KPL; ++j) pv[j] = sacc[kb][t * KPL + j];
          const V bv = pack_operand<V>(pv);
#pragma unroll
          for (int cb = 0; cb < D / 32; ++cb) {
            const T* vrow = vt + (cb * 32 + l32) * LY::VS + kb * 32;
            V av;
#pragma unroll
            for (int j = 0; j < KPL; ++j) vset(av, j, vrow[acc_row(t * KPL + j, hf)]);
            oacc[cb] = MF::run(av, bv, oacc[cb]);
          }
        }
    }

  }

  if constexpr (!LOGITS) {
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (qvalid) {
      const float inv = l_tot > 0.0f ? 1.0f / l_tot : 0.0f;
      T* orow = reinterpret_cast<T*>(a.out) + ((int64_t(b) * a.n_q + qi) * a.heads + h) * D;
#pragma unroll
      for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
        for (int i = 0; i < 16; ++i) orow[cb * 32 + acc_row(i, hf)] = T(oacc[cb][i] * inv);
      if (a.lse && hf == 0)
        a.lse[bh * a.n_q + qi] = l_tot > 0.0f ? m_run / sqrtf((float)D) + logf(l_tot) : -__builtin_inff();
    }
  }
}

template <typename T, int D>
size_t lds_bytes_t(int rank, int kc, bool tables) {
  size_t tile = 0;
  if (rank == 0) tile = Lds<T, D, 0>::tile_elems;
  else if (rank <= 16) tile = Lds<T, D, 16>::tile_elems;
  else tile = Lds<T, D, 32>::tile_elems;
  constexpr size_t TS = Lds<T, D, 0>::TS;
  return (2 * tile + (tables ? size_t(2) * kc * TS : 0)) * sizeof(T);  // two tile buffers
}

template <typename T, int D, int RP, bool LOGITS, bool TAB>
hipError_t launch_k(const AttendArgs& a, const dim3& grid, size_t lds, hipStream_t s) {
  const hipError_t e = hipFuncSetAttribute((const void*)attend_kernel<T, D, RP, LOGITS, TAB>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attend_kernel<T, D, RP, LOGITS, TAB>), grid, dim3(NT), lds, s, a);
  return hipGetLastError();
}

template <typename T, int D, int RP>
hipError_t launch_r(const AttendArgs& a, int batch, bool logits, hipStream_t s) {
  const dim3 grid((unsigned)((a.n_q + BQ - 1) / BQ), (unsigned)a.heads, (unsigned)batch);
  const bool tab = a.tables_in_lds != 0;
  const size_t lds = lds_bytes_t<T, D>(a.rank, a.n_centroids, tab);
  if (logits) return tab ? launch_k<T, D, RP, true, true>(a, grid, lds, s) : launch_k<T, D, RP, true, false>(a, grid, lds, s);
  return tab ? launch_k<T, D, RP, false, true>(a, grid, lds, s) : launch_k<T, D, RP, false, false>(a, grid, lds, s);
}

template <typename T, int D>
hipError_t launch_d(const AttendArgs& a, int batch, bool logits, hipStream_t s) {
  if (a.rank == 0) return launch_r<T, D, 0>(a, batch, logits, s);
  if (a.rank <= 16) return launch_r<T, D, 16>(a, batch, logits, s);
  return launch_r<T, D, 32>(a, batch, logits, s);
}

}  // namespace

constexpr size_t kLdsLimit = 160 * 1024;

size_t attend_lds_bytes(int d, int elem, int rank, int n_centroids, bool tables) {
  if (elem == 2) return d == 64 ? lds_bytes_t<bf16, 64>(rank, n_centroids, tables)
                                : lds_bytes_t<bf16, 128>(rank, n_centroids, tables);
  return d == 64 ? lds_bytes_t<float, 64>(rank, n_centroids, tables)
                 : lds_bytes_t<float, 128>(rank, n_centroids, tables);
}

bool attend_tables_fit(int d, int elem, int rank, int n_centroids) {
  return attend_lds_bytes(d, elem, rank, n_centroids, true) <= kLdsLimit;
}

hipError_t launch_attend_f32(const AttendArgs& a, int d, int batch, bool logits, hipStream_t s) {
  if (d == 64) return launch_d<float, 64>(a, batch, logits, s);
  if (d == 128) return launch_d<float, 128>(a, batch, logits, s);
  return hipErrorInvalidValue;
}

hipError_t launch_attend_bf16(const AttendArgs& a, int d, int batch, bool logits, hipStream_t s) {
  if (d == 64) return launch_d<bf16, 64>(a, batch, logits, s);
  if (d == 128) return launch_d<bf16, 128>(a, batch, logits, s);
  return hipErrorInvalidValue;
}

}  // namespace qwm
