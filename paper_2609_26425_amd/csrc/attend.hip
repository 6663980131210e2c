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

__device__ inline float bf16_bits_to_f(uint32_t hi16) { return __uint_as_float(hi16 << 16); }

constexpr int NW = 8, BQ = 32 * NW, KT = 64, NT = 64 * NW;

template <typename T, int D, int RP>
struct Lds {
  static constexpr int PK = sizeof(T) == 2 ? 8 : 1;  // row padding (elements)
  static constexpr int KS = D + PK;                  // K tile row stride
  static constexpr int CS = (RP > 0 ? RP : 1) + (sizeof(T) == 2 ? 4 : 1);
  static constexpr int VS = KT + PK;                 // V^T tile row stride
  static constexpr int tile_elems = KT * KS + KT * CS + D * VS;
};

template <typename T, int D, int RP, bool LOGITS>
__global__ __launch_bounds__(NT) void attend_kernel(const AttendArgs a) {
  typedef Mfma<T> MF;
  typedef typename MF::V V;
  constexpr int KPL = MF::KPL, KSTEP = MF::KSTEP;
  typedef Lds<T, D, RP> LY;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  T* smem = reinterpret_cast<T*>(smem_raw);
  const int Kc = a.n_centroids;
  T* tabK = smem;
  T* tabV = smem + (a.tables_in_lds ? Kc * D : 0);
  T* ktile = smem + (a.tables_in_lds ? 2 * Kc * D : 0);
  T* ctile = ktile + KT * LY::KS;
  T* vtile = ctile + KT * LY::CS;

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
  if (a.tables_in_lds) {
    const int n16 = Kc * D * int(sizeof(T)) / 16;
    const uint4* sk = reinterpret_cast<const uint4*>(gtabK);
    const uint4* sv = reinterpret_cast<const uint4*>(gtabV);
    uint4* dk = reinterpret_cast<uint4*>(tabK);
    uint4* dv = reinterpret_cast<uint4*>(tabV);
    for (int i = tid; i < n16; i += NT) { dk[i] = sk[i]; dv[i] = sv[i]; }
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

  const float kscale = 1.4426950408889634f / sqrtf((float)D);  // log2(e) / sqrt(d)
  float m_run = -__builtin_inff(), l_run = 0.0f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[cb][i] = 0.0f;

  constexpr int CHK = D * KT / NT;       // K channels per thread
  constexpr int CHV = D * KT / (2 * NT);  // V channels per thread (two keys)

  for (int64_t k0 = 0; k0 < kend; k0 += KT) {
    __syncthreads();
    // ---- dequantise the tile into LDS
    {  // Keys: thread -> (key, CHK consecutive channels inside one group)
      const int key = tid / (D / CHK), ch0 = (tid % (D / CHK)) * CHK;
      const int64_t tok = k0 + key;
      T* dst = ktile + key * LY::KS + ch0;
      if (tok < nc) {
        const int64_t slot = slot0 + tok;
        const int g = ch0 / G;
        int id = cache[L.k_ids + slot];
        id = id < Kc ? id : Kc - 1;
        const int z = (cache[L.k_zp + slot * L.zpb + g / 4] >> (2 * (g % 4))) & 3;
        const float s = (float)*reinterpret_cast<const _Float16*>(cache + L.k_scale + slot * 2 * L.ng + 2 * g);
        uint32_t cw;
        if constexpr (CHK == 16) cw = *reinterpret_cast<const uint32_t*>(cache + L.k_codes + slot * (D / 4) + ch0 / 4);
        else cw = *reinterpret_cast<const uint16_t*>(cache + L.k_codes + slot * (D / 4) + ch0 / 4);
        const T* mu = (a.tables_in_lds ? tabK : gtabK) + id * D + ch0;
#pragma unroll
        for (int c = 0; c < CHK; ++c) {
          const int q = (cw >> (2 * c)) & 3;
          dst[c] = T(__builtin_fmaf(s, (float)(q - z), (float)mu[c]));
        }
      } else {
#pragma unroll
        for (int c = 0; c < CHK; ++c) dst[c] = T(0.0f);
      }
    }
    if constexpr (RP > 0) {  // INT8 PSAC rows -> code * cscale
      constexpr int RCH = 8;
      if (tid < KT * (RP / RCH)) {
        const int key = tid / (RP / RCH), r0 = (tid % (RP / RCH)) * RCH;
        const int64_t tok = k0 + key;
        T* dst = ctile + key * LY::CS + r0;
        if (tok < nc) {
          const int64_t slot = slot0 + tok;
          const float cs = (float)*reinterpret_cast<const _Float16*>(cache + L.k_cscale + slot * 2);
          const int8_t* cp = reinterpret_cast<const int8_t*>(cache + L.k_coef + slot * r);
#pragma unroll
          for (int k = 0; k < RCH; ++k) dst[k] = T(r0 + k < r ? (float)cp[r0 + k] * cs : 0.0f);
        } else {
#pragma unroll
          for (int k = 0; k < RCH; ++k) dst[k] = T(0.0f);
        }
      }
    }
    {  // Values: thread -> (key pair, CHV channels), written transposed
      const int kp = tid % (KT / 2), ch0 = (tid / (KT / 2)) * CHV;
      float vv[2][CHV];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int64_t tok = k0 + 2 * kp + e;
        if (tok < nc) {
          const int64_t slot = slot0 + tok;
          const int g = ch0 / G;
          int id = cache[L.v_ids + slot];
          id = id < Kc ? id : Kc - 1;
          const int z = (cache[L.v_zp + slot * L.zpb + g / 4] >> (2 * (g % 4))) & 3;
          const float s = (float)*reinterpret_cast<const _Float16*>(cache + L.v_scale + slot * 2 * L.ng + 2 * g);
          uint32_t cw;
          if constexpr (CHV == 8) cw = *reinterpret_cast<const uint16_t*>(cache + L.v_codes + slot * (D / 4) + ch0 / 4);
          else cw = cache[L.v_codes + slot * (D / 4) + ch0 / 4];
          const T* mu = (a.tables_in_lds ? tabV : gtabV) + id * D + ch0;
#pragma unroll
          for (int c = 0; c < CHV; ++c) {
            const int q = (cw >> (2 * c)) & 3;
            vv[e][c] = __builtin_fmaf(s, (float)(q - z), (float)mu[c]);
          }
        } else {
#pragma unroll
          for (int c = 0; c < CHV; ++c) vv[e][c] = 0.0f;
        }
      }
#pragma unroll
      for (int c = 0; c < CHV; ++c) {
        T* dst = vtile + (ch0 + c) * LY::VS + 2 * kp;
        dst[0] = T(vv[0][c]);
        dst[1] = T(vv[1][c]);
      }
    }
    __syncthreads();

    // ---- logits tile S^T (keys x Queries) on matrix cores
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[kb][i] = 0.0f;
      const T* krow = ktile + (kb * 32 + l32) * LY::KS;
#pragma unroll
      for (int st = 0; st < D / KSTEP; ++st) {
        V av;
        if constexpr (KPL == 8) av = *reinterpret_cast<const V*>(krow + st * KSTEP + hf * KPL);
        else av = krow[st * KSTEP + hf];
        sacc[kb] = MF::run(av, qreg[st], sacc[kb]);
      }
      if constexpr (RP > 0) {
        const T* crow = ctile + (kb * 32 + l32) * LY::CS;
#pragma unroll
        for (int st = 0; st < RP / KSTEP; ++st) {
          V av;
#pragma unroll
          for (int j = 0; j < KPL; ++j) vset(av, j, crow[acc_row(st * KPL + j, hf)]);
          sacc[kb] = MF::run(av, ureg[st], sacc[kb]);
        }
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
      continue;
    }

    // ---- online softmax (base 2); masked keys -> -inf
    const bool need_mask = k0 + KT > kfull;
    float mt = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float v = sacc[kb][i] * kscale;
        if (need_mask && k0 + kb * 32 + acc_row(i, hf) >= lim) v = -__builtin_inff();
        sacc[kb][i] = v;
        mt = fmaxf(mt, v);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = m_new == -__builtin_inff() ? 0.0f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    m_run = m_new;
    float lsum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = __builtin_amdgcn_exp2f(sacc[kb][i] - m_use);
        sacc[kb][i] = p;
        lsum += p;
      }
    l_run = l_run * alpha + lsum;
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[cb][i] *= alpha;

    // ---- O^T += Vhat^T P^T (B operand = this lane's probabilities)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int t = 0; t < 32 / KSTEP; ++t) {
        V bv;
#pragma unroll
        for (int j = 0; j < KPL; ++j) vset(bv, j, T(sacc[kb][t * KPL + j]));
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb) {
          const T* vrow = vtile + (cb * 32 + l32) * LY::VS + kb * 32;
          V av;
#pragma unroll
          for (int j = 0; j < KPL; ++j) vset(av, j, vrow[acc_row(t * KPL + j, hf)]);
          oacc[cb] = MF::run(av, bv, oacc[cb]);
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
        a.lse[bh * a.n_q + qi] = l_tot > 0.0f ? m_run * 0.6931471805599453f + logf(l_tot) : -__builtin_inff();
    }
  }
}

template <typename T, int D>
size_t lds_bytes_t(int rank, int kc, bool tables) {
  size_t tile = 0;
  if (rank == 0) tile = Lds<T, D, 0>::tile_elems;
  else if (rank <= 16) tile = Lds<T, D, 16>::tile_elems;
  else tile = Lds<T, D, 32>::tile_elems;
  return (tile + (tables ? size_t(2) * kc * D : 0)) * sizeof(T);
}

template <typename T, int D, int RP>
hipError_t launch_r(const AttendArgs& a, int batch, bool logits, hipStream_t s) {
  const dim3 grid((unsigned)((a.n_q + BQ - 1) / BQ), (unsigned)a.heads, (unsigned)batch);
  const size_t lds = lds_bytes_t<T, D>(a.rank, a.n_centroids, a.tables_in_lds != 0);
  if (logits) {
    hipFuncSetAttribute((const void*)attend_kernel<T, D, RP, true>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL((attend_kernel<T, D, RP, true>), grid, dim3(NT), lds, s, a);
  } else {
    hipFuncSetAttribute((const void*)attend_kernel<T, D, RP, false>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL((attend_kernel<T, D, RP, false>), grid, dim3(NT), lds, s, a);
  }
  return hipGetLastError();
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
