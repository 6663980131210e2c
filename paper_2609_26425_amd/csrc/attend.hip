// Chunked attention over the packed 2-bit cache for gfx950 (Eq. 5 with the
// PSAC correction of Eq. 17), Keys and Values dequantised on chip.
//
// Per workgroup: one (b, h) and BQ = 256 Queries. The centroid tables of the
// head are staged in LDS once. For every 64-key tile four producer waves read
// the packed tile (codes, ids, zero-points, scales, INT8 coefficients) from HBM
// and rebuild
//     khat_0 = mu_z + s (q - z)   (Eq. 4, fp32, then the MFMA type)
//     chat   = code * cscale      (INT8 PSAC row)
//     vhat   = nu_z + s (q - z)
// into LDS (K row-major, V transposed, double-buffered), while eight consumer
// waves (32 Queries each) compute the previous tile's logits with matrix cores as S^T = [khat_0 | chat] [q | qU_r]^T over an augmented
// depth d + r, so (qU)c is added to qk^T before the softmax. With S^T each lane
// holds one Query column, so the exponentials feed the P.V product straight
// from the accumulator registers and O^T = Vhat^T P^T accumulates in registers.
// Softmax is online (running max and sum per Query, base-2 exponentials).
#include "attend_shape.h"
#include "xcd_order.h"

#include <atomic>
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

// max(a, b, c): the compiler folds the pair into one v_max3_f32. This file is
// built without NaN semantics (the logits and running maxima are finite or
// -inf), so no input is first quieted with a v_max_f32 x, x. It is not inline
// asm on purpose: its inputs come straight from matrix-core results, and only
// the compiler inserts the wait states a VALU read of those needs.
__device__ inline float max3f(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }

template <typename V>
__device__ inline auto vget(const V& v, int j) {
  if constexpr (std::is_same_v<V, float>) return v;
  else return v[j];
}

// Packed fields of one key tile held by one producer thread between their load
// and their dequantisation, as loaded (codes, centroid ids, zero-point bytes,
// binary16 scales), plus the active-chunk flags. Nothing is derived from a
// loaded value until the tile is dequantised, so the loads stay in flight.
// Marker: the coefficient-load form is chosen at run time.
struct AnyAlign {};

template <int NSUB>
struct TileRegs {
  uint32_t k_cw[NSUB], c_w[2], v_cw[2];
  uint32_t k_idb, v_idb[2];
  uint32_t k_zb[NSUB], v_zb[2];
  _Float16 k_s[NSUB], v_s[2], c_s;  // loaded bits, reinterpreted (no arithmetic)
  uint32_t k_cb[NSUB], v_cb[2];     // 8-bit group-scale codes (App. D.1 SI8 form only)
  bool k_on_act, v_on_act[2];
};

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

// N centroid components from LDS: BF16 (T), or with H16 the binary16 copy of
// the table (scaled by a power of two), which v_fma_mix_f32 converts to fp32 as
// an operand, so the dequant takes no separate unpack of a BF16 pair.
template <bool H16, typename T, int N>
__device__ inline void load_tab(const T* p, float (&out)[N]) {
  if constexpr (H16) {
    typedef _Float16 h8 __attribute__((ext_vector_type(8)));
    static_assert(N % 8 == 0, "binary16 table loads of 8 values");
#pragma unroll
    for (int i = 0; i < N / 8; ++i) {
      const h8 v = reinterpret_cast<const h8*>(p)[i];
#pragma unroll
      for (int k = 0; k < 8; ++k) out[8 * i + k] = (float)v[k];
    }
  } else {
    load_vals<T, N>(p, out);
  }
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

// max of x over lanes i and i ^ 32 (v_permlane32_swap: no LDS round trip)
__device__ inline float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// (x & m) | o in one v_and_or_b32; written as asm so that the compiler does not
// fold the mask into per-field extractions.
__device__ inline uint32_t and_or(uint32_t x, uint32_t m, uint32_t o) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(m), "v"(o));
  return r;
}

// x[c] = mu[c] + s (code_c - z) for the N consecutive channels of one code word
// (channel c in bits 2c). Each code is placed in a binary16 half as 1024 + code
// (exponent 10: one unit per ulp), so one packed f16 subtraction of 1024 + z
// yields two exact (code - z), and v_fma_mix_f32 takes them and the binary16
// scale as fp32 operands: one rounding, the same value as fma(s, code - z, mu).
// SI8 (App. D.1 8-bit group scales): the step is sigma * c with s = sigma and cm
// = (c, c); c (code - z) is an integer of magnitude <= 765, exact in binary16,
// so the fma still rounds once.
template <int N, bool SI8 = false, typename S>
__device__ inline void dequant_codes(uint32_t cw, S s, uint32_t zz, const float (&mu)[N], float (&x)[N],
                                     f16x2 cm = {}) {
  static_assert(N == 16 || N == 8, "16 or 8 channels per code word");
  const f16x2 zh = __builtin_bit_cast(f16x2, zz);
  // N == 8: channels 4..7 move to bits 16..23, so half k pairs channels k and k + N/2
  const uint32_t w = N == 16 ? cw : ((cw & 0xffu) | ((cw & 0xff00u) << 8));
#pragma unroll
  for (int k = 0; k < N / 2; ++k) {
    f16x2 d = __builtin_bit_cast(f16x2, and_or(w >> (2 * k), 0x00030003u, 0x64006400u)) - zh;
    if constexpr (SI8) d = d * cm;
    x[k] = __builtin_fmaf((float)s, (float)d.x, mu[k]);
    x[k + N / 2] = __builtin_fmaf((float)s, (float)d.y, mu[k + N / 2]);
  }
}

// N values of type T held as raw 32-bit words -> floats (exact).
template <typename T, int N>
__device__ inline void raw_to_float(const uint32_t* w, float (&x)[N]) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) x[i] = __uint_as_float(w[i]);
  }
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

// GEN: the launch has an exact active chunk after the packed keys and/or packed
// keys in several calibration epochs (a separate instance, so plain launches
// carry none of its code).
template <typename T, int D, int RP, bool LOGITS, bool TAB, bool GEN, bool SI8>
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

  // the wave index is uniform across a wave: taken through readfirstlane, the
  // producer/consumer split is a scalar branch, so neither role keeps the
  // other's registers live
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid / 64), lane = tid % 64, l32 = lane % 32,
            hf = lane / 32;
  // XCD-aware task order: workgroup L runs on XCD L % 8, so each XCD takes a
  // contiguous run of (Query block, head, batch) tasks, and the Query blocks
  // of a head, which stream the same key tiles at about the same time, read
  // them through one L2 instead of eight
  uint32_t bx, by, bz;
  {
    const uint32_t gx = gridDim.x, gy = gridDim.y, n = gx * gy * gridDim.z;
    const uint32_t L = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
    const uint32_t task = qwm_xcd_task(L, n);
    bx = task % gx;
    by = (task / gx) % gy;
    bz = task / (gx * gy);
  }
  const int h = int(by), b = int(bz);
  const int64_t bh = int64_t(b) * a.heads + h;
  // calibration slab of this head in epoch e
  auto epoch_slab = [&](int e) { return a.calib + int64_t(e) * a.calib_stride + bh * a.slab; };
  // epoch of a (wave-uniform) key, and the first key past epoch e
  // epoch of a key at or after the start of epoch e (epochs only advance with
  // the key, so the search starts from the last one found)
  auto epoch_from = [&](int e, int64_t key) {
    if constexpr (GEN)
      while (e + 1 < a.n_epochs && key >= a.epoch_start[e + 1]) ++e;
    return e;
  };
  auto epoch_at = [&](int64_t key) { return epoch_from(0, key); };
  auto epoch_end = [&](int e) -> int64_t {
    return GEN && e + 1 < a.n_epochs ? a.epoch_start[e + 1] : (int64_t(1) << 62);
  };
  auto epoch_begin = [&](int e) -> int64_t { return GEN ? a.epoch_start[e] : 0; };
  auto tab_of = [&](int e, int64_t off) { return reinterpret_cast<const T*>(epoch_slab(e) + off); };
  const CacheLayout& L = a.L;
  const uint8_t* cache = a.cache;
  const int64_t slot0 = bh * L.slots;
  const int r = a.rank;
  const int G = D / L.ng;
  const bool producer = wave >= NC;

  // ---- key range of this workgroup: Query block bx / n_split, and the
  // split-th of n_split equal runs of its key tiles
  // keys [0, npk) are packed; keys [npk, nc) are the exact active chunk
  const int64_t F = a.frame_tokens, qs = a.q_start, npk = a.n_cache, nc = a.n_cache + a.n_act;
  const int split = int(bx) % a.n_split;
  const int64_t qa = int64_t(bx / a.n_split) * BQ;
  const int64_t qb = qa + BQ < a.n_q ? qa + BQ : a.n_q;
  int64_t kend = LOGITS ? nc : qs + ((qb - 1) / F + 1) * F;
  if (kend > nc) kend = nc;
  // the logits hook may start its Queries at chunk row q_row0 (the mask's frame count)
  const int64_t qoff = LOGITS ? a.q_row0 : 0;
  int64_t kfull = qs + ((qa + qoff) / F + 1) * F;  // keys below are visible to every Query of the workgroup
  if (kfull > nc) kfull = nc;
  const int64_t ntile_all = (kend + KT - 1) / KT;
  // this launch covers tiles [tile_lo, ntile_all) (tile_lo is 0 unless the
  // caller splits the key range over launches)
  const int64_t tlo = a.tile_lo < ntile_all ? a.tile_lo : ntile_all;
  const int64_t per_split = (ntile_all - tlo + a.n_split - 1) / a.n_split;
  const int64_t t0 = tlo + split * per_split < ntile_all ? tlo + split * per_split : ntile_all;
  const int64_t ntile = t0 + per_split < ntile_all ? t0 + per_split : ntile_all;  // this split: tiles [t0, ntile)
  const int64_t nfull = npk / KT;  // tiles [0, nfull) hold packed keys only

  // ---- stage the centroid tables of one epoch (App. D.1: BF16 centroids) with
  // threads [first, first + count) of the workgroup
  // Plain BF16 instances stage the binary16 copies of the tables, which hold
  // mu 2^-e (e per table, from the calibration block): Keys and Values then
  // dequantise as mu 2^-e + (s 2^-e)(q - z), i.e. scaled by 2^-e exactly, and
  // the Query fragment (times 2^e_k) and the output (times 2^e_v) undo it, so
  // every product and sum of the attention is that of the BF16 tables.
  constexpr bool H16 = TAB && !GEN && sizeof(T) == 2;
  auto stage_tables = [&](int e, int first, int count) {
    constexpr int PER_ROW = D * int(sizeof(T)) / 16;  // 16-byte chunks per centroid row
    const uint4* sk = reinterpret_cast<const uint4*>(tab_of(e, H16 ? a.o_mu_k16 : a.o_mu_k));
    const uint4* sv = reinterpret_cast<const uint4*>(tab_of(e, H16 ? a.o_mu_v16 : a.o_mu_v));
    for (int i = tid - first; i < Kc * PER_ROW; i += count) {
      const int row = i / PER_ROW, ch = i % PER_ROW;
      *reinterpret_cast<uint4*>(tabK + row * LY::TS + ch * (16 / int(sizeof(T)))) = sk[i];
      *reinterpret_cast<uint4*>(tabV + row * LY::TS + ch * (16 / int(sizeof(T)))) = sv[i];
    }
  };
  // the staged epoch: that of the tile being dequantised (both roles track it)
  int se = epoch_at(t0 * KT);
  // 2^-e of the staged binary16 tables (1 without them)
  float sck = 1.0f, scv = 1.0f;
  int ek = 0, ev = 0;
  if constexpr (H16) {
    const int32_t* e16 = reinterpret_cast<const int32_t*>(epoch_slab(se) + a.o_e16);
    ek = e16[0];
    ev = e16[1];
    sck = ldexpf(1.0f, -ek);
    scv = ldexpf(1.0f, -ev);
  }
  if constexpr (TAB) stage_tables(se, 0, NT);

  // ======================= producer state (waves NC .. NC+NP-1)
  const int ptid = producer ? tid - NC * 64 : 0;
  constexpr int CHK = D * KT / PT;        // K channels per producer thread (one key)
  constexpr int NSUB = CHK / 16;          // 16-channel pieces
  constexpr int CHV = D * KT / (2 * PT);  // V channels per producer thread (two keys)
  constexpr int RCH = RP > 0 ? RP * KT / PT : 1;  // PSAC ranks per producer thread
  constexpr int RPT = RP > 0 ? RP / RCH : 1;
  const int kkey = ptid / (D / CHK), kch0 = (ptid % (D / CHK)) * CHK;
  const int vkp = ptid % (KT / 2), vch0 = (ptid / (KT / 2)) * CHV, vg = vch0 / G;
  const int ckey = ptid / RPT, cr0 = (ptid % RPT) * RCH;
  const bool crole = RP > 0 && cr0 < r;
  const bool raligned = r % RCH == 0;

  // packed tile fields of this thread: tile t sits in register set (t - t0) & 1,
  // so a tile's loads are issued two tiles ahead of its dequantisation
  TileRegs<NSUB> P0, P1;
  auto clear_regs = [&](TileRegs<NSUB>& p) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < NSUB; ++u) { p.k_cw[u] = 0; p.k_zb[u] = 0; p.k_s[u] = 0; p.k_cb[u] = 0; }
    p.c_w[0] = p.c_w[1] = 0;
    p.c_s = 0;
    p.k_idb = 0;
    p.k_on_act = false;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      p.v_cw[e] = 0; p.v_idb[e] = 0; p.v_zb[e] = 0; p.v_s[e] = 0; p.v_cb[e] = 0; p.v_on_act[e] = false;
    }
  };
  clear_regs(P0);
  clear_regs(P1);
  // keys of the active chunk are read in dequant itself (only the flags travel
  // from one tile to the next), so they cost no registers across the loop
  constexpr int KW = CHK * int(sizeof(T)) / 4, VW = CHV * int(sizeof(T)) / 4;
  const T* __restrict__ k_act = reinterpret_cast<const T*>(a.k_act);
  const T* __restrict__ v_act = reinterpret_cast<const T*>(a.v_act);
  const uint32_t npku = uint32_t(npk);
  // Packed fields are read with buffer loads: one resource per field of this
  // head (base = its first slot), this thread's byte offset inside a tile as the
  // vector offset (fixed for all tiles) and the tile's byte offset as the scalar
  // offset, so advancing a tile costs no vector instruction.
  // group-scale bytes per token: binary16 steps, or 8-bit codes (SI8)
  const uint32_t zpb = L.zpb, sstride = SI8 ? L.ng : 2 * L.ng, ncu = uint32_t(nc);
  // active-chunk row of key `key` (>= npk) at channel c0: [B, n_act, H, d]
  auto act_row = [&](const T* base, uint32_t key, int c0) {
    return base + ((int64_t(b) * a.n_act + (key - npku)) * a.heads + h) * D + c0;
  };
  auto load_words = [&](const T* src, uint32_t* w, int nw) {
    const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
    for (int i = 0; i < nw / 4; ++i) {
      const uint4 u = p[i];
      w[4 * i] = u.x; w[4 * i + 1] = u.y; w[4 * i + 2] = u.z; w[4 * i + 3] = u.w;
    }
  };
  auto field = [&](int64_t off, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)(cache + off + slot0 * bytes), 0,
                                             int(uint32_t(L.slots) * bytes), 0x00020000);
  };
  const auto r_kc = field(L.k_codes, D / 4), r_ki = field(L.k_ids, 1), r_kz = field(L.k_zp, zpb),
             r_ks = field(L.k_scale, sstride), r_vc = field(L.v_codes, D / 4), r_vi = field(L.v_ids, 1),
             r_vz = field(L.v_zp, zpb), r_vs = field(L.v_scale, sstride);
  const auto r_cc = field(L.k_coef, uint32_t(r)), r_cs = field(L.k_cscale, 2);
  // sparse rows (general instance only): this head's row pool and tile directory
  const auto r_pc = __builtin_amdgcn_make_buffer_rsrc((void*)(cache + L.k_coef + bh * L.pool * r), 0,
                                                      int(uint32_t(L.pool) * uint32_t(r)), 0x00020000);
  const auto r_ps = __builtin_amdgcn_make_buffer_rsrc((void*)(cache + L.k_cscale + bh * L.pool * 2), 0,
                                                      int(uint32_t(L.pool) * 2u), 0x00020000);
  const uint32_t* dir = reinterpret_cast<const uint32_t*>(cache + L.k_dir + bh * (L.slots / 64) * 16);
  const auto r_ksg = field(L.k_sigma, 2), r_vsg = field(L.v_sigma, 2);  // SI8 secondary scales
  const int o_kc = kkey * (D / 4) + kch0 / 4, o_kz = kkey * zpb, o_ks = kkey * sstride;
  const int o_cc = ckey * r + cr0, o_cs = ckey * 2;
  const int o_vc = 2 * vkp * (D / 4) + vch0 / 4, o_vz = 2 * vkp * zpb + vg / 4,
            o_vs = 2 * vkp * sstride + (SI8 ? vg : 2 * vg);

  // FULL: every key of the tile is < n_cache, so no per-thread guards. A key
  // past n_cache (tail tiles only) gets centroid 0, scale 0 and code 0: a finite
  // placeholder whose logit the mask turns into -inf, so it never contributes.
  // residual group, zero-point byte and 2-bit shift of each K piece and of the V run
  int kgrp[NSUB];
#pragma unroll
  for (int u = 0; u < NSUB; ++u) kgrp[u] = (kch0 + 16 * u) / G;
  const int vzsh = 2 * (vg % 4);
  // Placeholder fields (all zero) decode to centroid 0 with scale 0.
  // align_tag: std::true_type / std::false_type when the caller knows whether
  // r is a multiple of RCH (one whole-word coefficient load), else AnyAlign
  auto load_raw = [&](TileRegs<NSUB>& p, auto full_tag, uint32_t k0, auto align_tag) __attribute__((always_inline)) {
    constexpr bool FULL = decltype(full_tag)::value;
    using AT = decltype(align_tag);
    constexpr int AL = std::is_same_v<AT, std::true_type> ? 1 : std::is_same_v<AT, std::false_type> ? 0 : -1;
    const bool aligned = AL == 1 || (AL == -1 && raligned);
    const int k0i = int(k0);
    // fields are gathered in locals and stored into the set once, at the end
    uint32_t kid = 0, kzb[NSUB], kcw[NSUB], kcb[NSUB], cw2[2] = {0, 0};
    uint32_t vid[2] = {0, 0}, vzb[2] = {0, 0}, vcw[2] = {0, 0}, vcb[2] = {0, 0};
    _Float16 ksb[NSUB], csb = 0, vsb[2] = {0, 0};
#pragma unroll
    for (int u = 0; u < NSUB; ++u) { kzb[u] = 0; ksb[u] = 0; kcw[u] = 0; kcb[u] = 0; }
    const bool kact = GEN && !FULL && k0 + kkey >= npku && k0 + kkey < ncu;
    if (!kact && (FULL || k0 + kkey < npku)) {
      kid = __builtin_amdgcn_raw_buffer_load_b8(r_ki, kkey, k0i, 0);
#pragma unroll
      for (int u = 0; u < NSUB; ++u) {
        const int g = kgrp[u];
        kzb[u] = __builtin_amdgcn_raw_buffer_load_b8(r_kz, o_kz + g / 4, k0i * int(zpb), 0);
        if constexpr (SI8) kcb[u] = __builtin_amdgcn_raw_buffer_load_b8(r_ks, o_ks + g, k0i * int(sstride), 0);
        else ksb[u] = __builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(r_ks, o_ks + 2 * g, k0i * int(sstride), 0));
      }
      if constexpr (SI8) {
        const _Float16 sg = __builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(r_ksg, 2 * kkey, k0i * 2, 0));
#pragma unroll
        for (int u = 0; u < NSUB; ++u) ksb[u] = sg;
      }
      if constexpr (NSUB == 2) {
        const auto cw = __builtin_amdgcn_raw_buffer_load_b64(r_kc, o_kc, k0i * (D / 4), 0);
        kcw[0] = cw[0];
        kcw[1] = cw[1];
      } else {
        kcw[0] = __builtin_amdgcn_raw_buffer_load_b32(r_kc, o_kc, k0i * (D / 4), 0);
      }
    }
    if constexpr (RP > 0) {
      if (GEN && L.sparse && crole && (FULL || k0 + ckey < npku)) {
        // the key's row through the directory entry of its 64-key tile: present
        // iff its mask bit is set, at pool row base + (set bits below it)
        const uint32_t* e = dir + (k0 / 64) * 4;
        const uint64_t m = uint64_t(e[2]) | (uint64_t(e[3]) << 32);
        if ((m >> ckey) & 1) {
          const int row = int(e[0]) + __popcll(m & ((uint64_t(1) << ckey) - 1));
          csb = __builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(r_ps, row * 2, 0, 0));
#pragma unroll
          for (int k = 0; k < RCH; ++k)
            if (cr0 + k < r)
              cw2[k / 4] |= uint32_t(__builtin_amdgcn_raw_buffer_load_b8(r_pc, row * r + cr0 + k, 0, 0)) << (8 * (k % 4));
        }
      } else if (crole && (FULL || k0 + ckey < npku)) {
        csb = __builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(r_cs, o_cs, k0i * 2, 0));
        if (aligned) {
          if constexpr (RCH == 8) {
            const auto u = __builtin_amdgcn_raw_buffer_load_b64(r_cc, o_cc, k0i * r, 0);
            cw2[0] = u[0];
            cw2[1] = u[1];
          } else {
            cw2[0] = __builtin_amdgcn_raw_buffer_load_b32(r_cc, o_cc, k0i * r, 0);
          }
        } else {
#pragma unroll
          for (int k = 0; k < RCH; ++k)
            if (cr0 + k < r) cw2[k / 4] |= uint32_t(__builtin_amdgcn_raw_buffer_load_b8(r_cc, o_cc + k, k0i * r, 0)) << (8 * (k % 4));
        }
      }
    }
    bool vact[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const uint32_t key = k0 + 2 * vkp + e;
      vact[e] = GEN && !FULL && key >= npku && key < ncu;
      if (!vact[e] && (FULL || key < npku)) {
        vid[e] = __builtin_amdgcn_raw_buffer_load_b8(r_vi, 2 * vkp + e, k0i, 0);
        vzb[e] = __builtin_amdgcn_raw_buffer_load_b8(r_vz, o_vz + e * int(zpb), k0i * int(zpb), 0);
        if constexpr (SI8) {
          vcb[e] = __builtin_amdgcn_raw_buffer_load_b8(r_vs, o_vs + e * int(sstride), k0i * int(sstride), 0);
          vsb[e] = __builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(r_vsg, 2 * (2 * vkp + e), k0i * 2, 0));
        } else {
          vsb[e] = __builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(r_vs, o_vs + e * int(sstride), k0i * int(sstride), 0));
        }
        if constexpr (CHV == 16) vcw[e] = __builtin_amdgcn_raw_buffer_load_b32(r_vc, o_vc + e * (D / 4), k0i * (D / 4), 0);
        else vcw[e] = __builtin_amdgcn_raw_buffer_load_b16(r_vc, o_vc + e * (D / 4), k0i * (D / 4), 0);
      }
    }
    p.k_on_act = kact;
    p.k_idb = kid;
#pragma unroll
    for (int u = 0; u < NSUB; ++u) { p.k_zb[u] = kzb[u]; p.k_s[u] = ksb[u]; p.k_cw[u] = kcw[u]; p.k_cb[u] = kcb[u]; }
    p.c_s = csb;
    p.c_w[0] = cw2[0];
    p.c_w[1] = cw2[1];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      p.v_on_act[e] = vact[e]; p.v_idb[e] = vid[e]; p.v_zb[e] = vzb[e]; p.v_s[e] = vsb[e]; p.v_cw[e] = vcw[e];
      p.v_cb[e] = vcb[e];
    }
  };

  // rebuild khat_0 = mu + s (q - z) (Eq. 4), chat = code * cscale and vhat into
  // tile buffer `buf`. s (q - z) is exact in fp32, so the fma rounds once,
  // exactly like mu + s (q - z).
  auto dequant_tile = [&](TileRegs<NSUB>& p, auto full_tag, int64_t t) __attribute__((always_inline)) {
    // FULL: every key of the tile is packed, so no active-chunk branch
    constexpr bool FULL = decltype(full_tag)::value;
    const uint32_t (&k_cw)[NSUB] = p.k_cw;
    const uint32_t (&c_w)[2] = p.c_w;
    const uint32_t (&v_cw)[2] = p.v_cw;
    const bool k_on_act = p.k_on_act, v_on_act[2] = {p.v_on_act[0], p.v_on_act[1]};
    // fields as the decode takes them: clamped ids, (1024 + z) pairs, binary16 scales
    const int k_id = int(p.k_idb) < Kc ? int(p.k_idb) : Kc - 1;
    uint32_t k_z[NSUB], v_z[2];
    // steps as loaded (binary16), or scaled by 2^-e (fp32) with the binary16 tables
    std::conditional_t<H16, float, _Float16> k_s[NSUB], v_s[2];
    int v_id[2];
#pragma unroll
    for (int u = 0; u < NSUB; ++u) {
      k_z[u] = (0x6400u + ((p.k_zb[u] >> (2 * (kgrp[u] % 4))) & 3)) * 0x00010001u;
      if constexpr (H16) k_s[u] = (float)p.k_s[u] * sck;  // exact: a power of two
      else k_s[u] = p.k_s[u];
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      v_id[e] = int(p.v_idb[e]) < Kc ? int(p.v_idb[e]) : Kc - 1;
      v_z[e] = (0x6400u + ((p.v_zb[e] >> vzsh) & 3)) * 0x00010001u;
      if constexpr (H16) v_s[e] = (float)p.v_s[e] * scv;
      else v_s[e] = p.v_s[e];
    }
    const float c_s = (float)p.c_s;
    const int buf = int(t & 1);
    const uint32_t k0 = uint32_t(t * KT);
    T* kt = smem + tile0 + buf * LY::tile_elems;
    T* ct = kt + KT * LY::KS;
    T* vt = ct + KT * LY::CS;
    // centroids: the staged epoch se (LDS tables when they fit); a tile may end in
    // the next epoch, whose keys read that epoch's tables from global memory
    const int64_t b1 = epoch_end(se);
    const int se1 = se + 1 < a.n_epochs ? se + 1 : se;
    const T* gK0 = tab_of(se, a.o_mu_k);
    const T* gK1 = tab_of(se1, a.o_mu_k);
    const T* gV0 = tab_of(se, a.o_mu_v);
    const T* gV1 = tab_of(se1, a.o_mu_v);
    const bool k_e1 = GEN && !FULL && int64_t(k0) + kkey >= b1;
    bool v_e1[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) v_e1[e] = GEN && !FULL && int64_t(k0) + 2 * vkp + e >= b1;
#pragma unroll
    for (int u = 0; u < NSUB; ++u) {
      float mu[16], x[16];
      if (TAB && !k_e1) load_tab<H16, T, 16>(tabK + k_id * LY::TS + kch0 + 16 * u, mu);
      else load_vals<T, 16>((k_e1 ? gK1 : gK0) + k_id * D + kch0 + 16 * u, mu);
      if (GEN && !FULL && k_on_act) {
        uint32_t w[16 * sizeof(T) / 4];
        load_words(act_row(k_act, k0 + kkey, kch0 + 16 * u), w, 16 * int(sizeof(T)) / 4);
        raw_to_float<T, 16>(w, x);
      } else {
        const _Float16 cb = (_Float16)p.k_cb[u];
        dequant_codes<16, SI8>(k_cw[u], k_s[u], k_z[u], mu, x, f16x2{cb, cb});
      }
      store_vals<T, 16>(kt + kkey * LY::KS + kch0 + 16 * u, x);
    }
    if constexpr (RP > 0) {
      if (ptid < KT * RPT) {
        float x[RCH];
#pragma unroll
        for (int k = 0; k < RCH; ++k) x[k] = (float)int8_t((c_w[k / 4] >> (8 * (k % 4))) & 255) * c_s;
        store_vals8<T, RCH>(ct + ckey * LY::CS + cr0, x);
      }
    }
    {
      float x0[CHV], x1[CHV];
      float mu0[CHV], mu1[CHV];
      const _Float16 vc0 = (_Float16)p.v_cb[0], vc1 = (_Float16)p.v_cb[1];
      const f16x2 vcm0 = {vc0, vc0}, vcm1 = {vc1, vc1};
      if (TAB && !v_e1[0]) load_tab<H16, T, CHV>(tabV + v_id[0] * LY::TS + vch0, mu0);
      else load_vals<T, CHV>((v_e1[0] ? gV1 : gV0) + v_id[0] * D + vch0, mu0);
      if (TAB && !v_e1[1]) load_tab<H16, T, CHV>(tabV + v_id[1] * LY::TS + vch0, mu1);
      else load_vals<T, CHV>((v_e1[1] ? gV1 : gV0) + v_id[1] * D + vch0, mu1);
      if (GEN && !FULL && (v_on_act[0] || v_on_act[1])) {
        uint32_t w[VW];
        if (v_on_act[0]) {
          load_words(act_row(v_act, k0 + 2 * vkp, vch0), w, VW);
          raw_to_float<T, CHV>(w, x0);
        } else {
          dequant_codes<CHV, SI8>(v_cw[0], v_s[0], v_z[0], mu0, x0, vcm0);
        }
        if (v_on_act[1]) {
          load_words(act_row(v_act, k0 + 2 * vkp + 1, vch0), w, VW);
          raw_to_float<T, CHV>(w, x1);
        } else {
          dequant_codes<CHV, SI8>(v_cw[1], v_s[1], v_z[1], mu1, x1, vcm1);
        }
      } else {
        dequant_codes<CHV, SI8>(v_cw[0], v_s[0], v_z[0], mu0, x0, vcm0);
        dequant_codes<CHV, SI8>(v_cw[1], v_s[1], v_z[1], mu1, x1, vcm1);
      }
#pragma unroll
      for (int c = 0; c < CHV; ++c) store_pair<T>(vt + (vch0 + c) * LY::VS + 2 * vkp, x0[c], x1[c]);
    }
  };

  using Full = std::integral_constant<bool, true>;
  using Tail = std::integral_constant<bool, false>;

  auto prefetch = [&](TileRegs<NSUB>& p, int64_t t) __attribute__((always_inline)) {
    if (t < nfull) load_raw(p, Full{}, uint32_t(t * KT), AnyAlign{});
    else load_raw(p, Tail{}, uint32_t(t * KT), AnyAlign{});
  };

  // ======================= consumer state (waves 0 .. NC-1)
  // Query and key positions fit in 32 bits (the host rejects larger calls)
  const int qi = int(qa) + (producer ? 0 : wave) * 32 + l32;
  const bool qvalid = !producer && qi < a.n_q;
  // a consumer wave of the last Query block whose 32 Queries all lie past n_q
  // (wave-uniform): it keeps the barriers of every tile and computes nothing
  const bool idle = !producer && qa + int64_t(wave) * 32 >= a.n_q;
  V qreg[D / KSTEP];
  V ureg[RP > 0 ? RP / KSTEP : 1];   // q U_r of epoch ue
  int ue = se;
  // u = q U_r of epoch e on matrix cores (A operand: rows = ranks of U_r^T);
  // every lane takes part, so callers stay wave-uniform
  auto compute_u = [&](int e, V (&dst)[RP > 0 ? RP / KSTEP : 1]) {
    const T* gU = tab_of(e, a.o_u_t);
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
    for (int st = 0; st < (RP > 0 ? RP / KSTEP : 1); ++st)
#pragma unroll
      for (int j = 0; j < KPL; ++j) vset(dst[st], j, T(uacc[st * KPL + j]));
  };
  float m_run = -__builtin_inff(), l_run = 0.0f;
  f32x16 oacc[D / 32];
  int lim = int(nc);
  if (!producer) {
    // Query fragment (B operand: k = channel, column = Query)
    const T* qrow = reinterpret_cast<const T*>(a.q) + ((int64_t(b) * a.n_q + (qvalid ? qi : 0)) * a.heads + h) * D;
#pragma unroll
    for (int st = 0; st < D / KSTEP; ++st) {
#pragma unroll
      for (int j = 0; j < KPL; ++j) vset(qreg[st], j, qvalid ? qrow[st * KSTEP + hf * KPL + j] : T(0.0f));
    }
    if constexpr (RP > 0) compute_u(se, ureg);
    if constexpr (H16) {
      // q 2^e_k (exact in BF16) against the Keys scaled by 2^-e_k
#pragma unroll
      for (int st = 0; st < D / KSTEP; ++st)
#pragma unroll
        for (int j = 0; j < KPL; ++j) vset(qreg[st], j, T(ldexpf(float(vget(qreg[st], j)), ek)));
    }
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[cb][i] = 0.0f;
    if (qvalid) {
      const int64_t l = qs + ((qi + qoff) / F + 1) * F;  // this lane's Query sees keys j < lim
      lim = int(l < nc ? l : nc);
    }
  }
  const float mscale = 1.4426950408889634f / sqrtf((float)D);  // logits are exponentiated as 2^(S log2(e)/sqrt(d))

  // Producers and consumers run separate loops with one barrier per tile each,
  // so neither keeps the other's registers live.
  // Every thread staged part of the centroid tables: they must be complete
  // before the first dequantisation. The producers' first packed loads are
  // already in flight across this barrier.
  if (producer && t0 < ntile) {
    prefetch(P0, t0);
    if (t0 + 1 < ntile) prefetch(P1, t0 + 1);
  }
  if constexpr (TAB) __syncthreads();

  if (producer) {
    // Producers issue first: their vector work fills the matrix-core phases of
    // the consumers, and a late tile would stall all eight consumers.
    __builtin_amdgcn_s_setprio(2);
    if (t0 < ntile) {
      dequant_tile(P0, Tail{}, t0);  // the general form is right for any tile
      if (t0 + 2 < ntile) prefetch(P0, t0 + 2);
    }
    // One step per key tile `it`, after its barrier (buffer it&1 is complete and
    // every consumer is done with buffer (it+1)&1): dequantise tile it + 1 from
    // its register set, then refill that set with tile it + 3. Every call names
    // its set statically (a set chosen at run time would be kept in memory).
    auto refill = [&](TileRegs<NSUB>& p, int64_t it, auto full_tag) __attribute__((always_inline)) {
      dequant_tile(p, full_tag, it + 1);
      if (it + 3 < ntile) prefetch(p, it + 3);
    };
    // The steady loops take two tiles per trip with the sets in fixed places, so
    // the wait before each dequantisation covers only the older set's loads.
    if constexpr (GEN) {
      auto gstep = [&](int64_t it, TileRegs<NSUB>& p) __attribute__((always_inline)) {
        __syncthreads();
        if constexpr (TAB) {
          // the next tile opens another epoch: restage its tables (every producer
          // is done with the old ones after the barrier above), then sync
          if (it + 1 < ntile) {
            const int en = epoch_from(se, (it + 1) * KT);
            if (en != se) {
              se = en;
              stage_tables(se, NC * 64, PT);
              __syncthreads();
            }
          }
        } else {
          if (it + 1 < ntile) se = epoch_from(se, (it + 1) * KT);
        }
        if (it + 1 < ntile) {
          // a tile of packed keys inside one epoch takes the plain form
          const int64_t kn = (it + 1) * KT;
          if (kn + KT <= npk && kn + KT <= epoch_end(se)) refill(p, it, Full{});
          else refill(p, it, Tail{});
        }
      };
      int64_t it = t0;
      for (; it + 1 < ntile; it += 2) {
        gstep(it, P1);
        gstep(it + 1, P0);
      }
      if (it < ntile) gstep(it, P1);
      return;
    }
    // Steady state: the dequantised tile and the prefetched one (it + 3) are both
    // all packed, so every load is issued unconditionally and the loads of one
    // set stay in flight across the other set's dequantisation. The loop is
    // compiled once per coefficient-load form.
    const int64_t nsteady = (nfull < ntile ? nfull : ntile) - 3;  // it < nsteady: it + 3 < min(nfull, ntile)
    int64_t it = t0;
    auto steady = [&](auto align_tag) __attribute__((always_inline)) {
      for (; it + 1 < nsteady; it += 2) {
        __syncthreads();
        dequant_tile(P1, Full{}, it + 1);
        load_raw(P1, Full{}, uint32_t((it + 3) * KT), align_tag);
        __syncthreads();
        dequant_tile(P0, Full{}, it + 2);
        load_raw(P0, Full{}, uint32_t((it + 4) * KT), align_tag);
      }
    };
    if (raligned) steady(std::true_type{});
    else steady(std::false_type{});
    // the last steps (it - t0 is even here) in the general form
    for (; it < ntile; it += 2) {
      __syncthreads();
      if (it + 1 < ntile) refill(P1, it, Tail{});
      if (it + 1 < ntile) {
        __syncthreads();
        if (it + 2 < ntile) refill(P0, it + 1, Tail{});
      }
    }
    return;
  }

  // Lazy rescaling: the running max m_run is raised only when a logit exceeds it
  // by more than tau (2^8 in probability), so probabilities stay below 256 and
  // the rescale of O is rare after the first tiles. O / l and lse are exact for
  // any m_run, so this changes no result beyond rounding.
  const float tau = 8.0f / mscale;

  // Tiles below kfull need no mask: they run as a separate instance of the tile
  // code without the mask branches, so nothing splits its instruction stream.
  auto tile = [&](int64_t it, auto mask_tag) {
    constexpr bool MASKED = decltype(mask_tag)::value;
    const int64_t k0 = it * KT;
    __syncthreads();
    if constexpr (GEN && TAB) {
      // mirror of the producers' restage of the centroid tables (one more barrier)
      if (it + 1 < ntile) {
        const int en = epoch_from(se, (it + 1) * KT);
        if (en != se) {
          se = en;
          __syncthreads();
        }
      }
    }
    if (idle) return;
    const T* kt = smem + tile0 + int(it & 1) * LY::tile_elems;
    const T* ct = kt + KT * LY::KS;
    const T* vt = ct + KT * LY::CS;
    // PSAC terms use q U_r of the key's epoch (ureg holds that of epoch ue): the
    // tile's first epoch here, and where a half crosses into the next epoch at
    // b1, u is recomputed for it in the middle of that half's product
    int64_t b1 = int64_t(1) << 62;
    if constexpr (GEN && RP > 0) {
      const int e0 = epoch_from(ue, k0);
      if (e0 != ue) {
        compute_u(e0, ureg);
        ue = e0;
      }
      b1 = epoch_end(e0) < npk ? epoch_end(e0) : (int64_t(1) << 62);
    }

    // logits S^T of the 32 keys k0 + 32 kb + row (rows x Queries) on matrix cores
    auto k_part = [&](f32x16 acc, int kb) __attribute__((always_inline)) {
      const T* krow = kt + (kb * 32 + l32) * LY::KS;
#pragma unroll
      for (int st = 0; st < D / KSTEP; ++st) {
        V av;
        if constexpr (KPL == 8) av = *reinterpret_cast<const V*>(krow + st * KSTEP + hf * KPL);
        else av = krow[st * KSTEP + hf];
        acc = MF::run(av, qreg[st], acc);
      }
      return acc;
    };
    auto logits_half = [&](int kb) {
      f32x16 acc;
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
      if constexpr (RP > 0) {
        const T* crow = ct + (kb * 32 + l32) * LY::CS;
        V av[RP / KSTEP];
#pragma unroll
        for (int st = 0; st < RP / KSTEP; ++st)
#pragma unroll
          for (int j = 0; j < KPL; ++j) vset(av[st], j, crow[acc_row(st * KPL + j, hf)]);
        const int64_t h0 = k0 + kb * 32;
        if (GEN && b1 >= h0 && b1 < h0 + 32) {
          // the half crosses into the next epoch: this lane's A row is key
          // h0 + l32, whose chat goes with its own epoch's u. u of the next
          // epoch is computed first, while no accumulator is live, and the PSAC
          // term goes in before q . khat_0
          V un[RP > 0 ? RP / KSTEP : 1];
          compute_u(ue + 1, un);
          const bool first = h0 + l32 < b1;
#pragma unroll
          for (int st = 0; st < RP / KSTEP; ++st) {
            V a0, a1;
#pragma unroll
            for (int j = 0; j < KPL; ++j) {
              vset(a0, j, first ? vget(av[st], j) : T(0.0f));
              vset(a1, j, first ? T(0.0f) : vget(av[st], j));
            }
            acc = MF::run(a0, ureg[st], acc);
            acc = MF::run(a1, un[st], acc);
          }
#pragma unroll
          for (int st = 0; st < RP / KSTEP; ++st) ureg[st] = un[st];
          ue = ue + 1;
          return k_part(acc, kb);
        }
        acc = k_part(acc, kb);
#pragma unroll
        for (int st = 0; st < RP / KSTEP; ++st) acc = MF::run(av[st], ureg[st], acc);
        return acc;
      }
      return k_part(acc, kb);
    };

    if constexpr (LOGITS) {
      const float inv = 1.0f / sqrtf((float)D);
      float* lrow = a.logits + (bh * a.n_q + (qvalid ? qi : 0)) * nc;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        // every lane takes part in the matrix-core product: its operand reads
        // feed the whole wave, so they may not sit under a per-lane condition
        const f32x16 sv = logits_half(kb);
        if (qvalid) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int64_t j = k0 + kb * 32 + acc_row(i, hf);
            if (j < nc) lrow[j] = j < lim ? sv[i] * inv : -__builtin_inff();
          }
        }
      }
    } else {
      // masked keys (only in tiles past kfull, and a first tile that starts
      // below key_lo) -> -inf
      auto mask_half = [&](f32x16& sv, int kb) {
        if constexpr (MASKED) {
          const int klo = int(a.key_lo);
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = int(k0) + kb * 32 + acc_row(i, hf);
            if (key >= lim || key < klo) sv[i] = -__builtin_inff();
          }
        }
      };
      // raise m_run if the max over these 32 keys exceeds it by more than tau
      auto raise_max = [&](const f32x16& sv) {
        float mt = -__builtin_inff();
#pragma unroll
        for (int i = 0; i < 8; ++i) mt = max3f(mt, sv[2 * i], sv[2 * i + 1]);
        mt = max_halves(mt);
        if (__any(mt > m_run + tau)) {
          const float m_new = fmaxf(m_run, mt);
          const float alpha = m_new == -__builtin_inff() ? 1.0f : __builtin_amdgcn_exp2f((m_run - m_new) * mscale);
          l_run *= alpha;
#pragma unroll
          for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
            for (int i = 0; i < 16; ++i) oacc[cb][i] *= alpha;
          m_run = m_new;
        }
      };
      auto probs = [&](f32x16& sv) {
        const float mc = m_run == -__builtin_inff() ? 0.0f : -m_run * mscale;
#pragma unroll
        for (int i = 0; i < 16; ++i) sv[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[i], mscale, mc));
        if constexpr (KPL == 1) {
          float lpart[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int i = 0; i < 16; ++i) lpart[i % 4] += sv[i];
          l_run += (lpart[0] + lpart[1]) + (lpart[2] + lpart[3]);
        }
      };
      // O^T += Vhat^T P^T over the 32 keys of half kb (B operand = this lane's probabilities)
      auto pv_half = [&](const f32x16& pv32, int kb) {
#pragma unroll
        for (int t = 0; t < 32 / KSTEP; ++t) {
          float pv[KPL];
#pragma unroll
          for (int j = 0; j < KPL; ++j) pv[j] = pv32[t * KPL + j];
          const V bv = pack_operand<V>(pv);
          if constexpr (KPL == 8) {
            // row sum of the probabilities as rounded for the product: two per v_dot2_f32_bf16
            const bf16x2 one = {bf16(1.0f), bf16(1.0f)};
            const uint4 pw = __builtin_bit_cast(uint4, bv);
            const uint32_t w[4] = {pw.x, pw.y, pw.z, pw.w};
#pragma unroll
            for (int j = 0; j < 4; ++j)
              l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[j]), one, l_run, false);
          }
#pragma unroll
          for (int cb = 0; cb < D / 32; ++cb) {
            const T* vrow = vt + (cb * 32 + l32) * LY::VS + kb * 32;
            V av;
#pragma unroll
            for (int j = 0; j < KPL; ++j) vset(av, j, vrow[acc_row(t * KPL + j, hf)]);
            oacc[cb] = MF::run(av, bv, oacc[cb]);
          }
        }
      };

      if constexpr (!GEN) {
        // the tile's two halves of 32 keys: the second half's logits products
        // are issued before the first half's exponentials, which need none of
        // them, so the matrix cores run while the vector unit computes
        // probabilities. The running max of the second half is raised only
        // after the first half's P V is in O (a rescale must cover it).
        f32x16 s0 = logits_half(0);
        mask_half(s0, 0);
        raise_max(s0);
        f32x16 s1 = logits_half(1);
        probs(s0);
        pv_half(s0, 0);
        mask_half(s1, 1);
        raise_max(s1);
        probs(s1);
        pv_half(s1, 1);
      } else {
        // streaming forms: one half at a time (the epoch-crossing path of the
        // logits leaves no room for a second live half)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          f32x16 sv = logits_half(kb);
          mask_half(sv, kb);
          raise_max(sv);
          probs(sv);
          pv_half(sv, kb);
        }
      }
    }
  };
  const int64_t nclean = kfull / KT < ntile ? kfull / KT : ntile;
  int64_t it = t0;
  if (it < ntile && a.key_lo > it * KT) {  // the first tile holds keys below key_lo
    tile(it, std::integral_constant<bool, true>{});
    ++it;
  }
  for (; it < nclean; ++it) tile(it, std::integral_constant<bool, false>{});
  for (; it < ntile; ++it) tile(it, std::integral_constant<bool, true>{});

  if constexpr (!LOGITS) {
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (a.n_split > 1 || a.partial) {
      // partial result of this split: unnormalised O, the running max (raw logit
      // units) and the sum; attend_combine merges the splits
      if (qvalid) {
        const int64_t row = (int64_t(a.split_base + split) * a.heads * gridDim.z + bh) * a.n_q + qi;
        float* po = a.part_o + row * D;
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
          for (int i = 0; i < 16; ++i) po[cb * 32 + acc_row(i, hf)] = H16 ? ldexpf(oacc[cb][i], ev) : oacc[cb][i];
        if (hf == 0) {
          a.part_ml[2 * row] = m_run;
          a.part_ml[2 * row + 1] = l_tot;
        }
      }
    } else {
      if (qvalid) {
        // O / l; with the binary16 tables, times 2^e_v (the Values were scaled by 2^-e_v)
        const float inv = l_tot > 0.0f ? (H16 ? ldexpf(1.0f / l_tot, ev) : 1.0f / l_tot) : 0.0f;
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
}

template <typename T, int D, int RP, bool LOGITS, bool TAB, bool GEN = false, bool SI8 = false>
hipError_t launch_k(const AttendArgs& a, const dim3& grid, size_t lds, hipStream_t s) {
  // the dynamic LDS limit is raised once per device for this instance
  static std::atomic<uint64_t> raised{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? uint64_t(1) << dev : 0;
  if (!bit || !(raised.load(std::memory_order_acquire) & bit)) {
    e = hipFuncSetAttribute((const void*)attend_kernel<T, D, RP, LOGITS, TAB, GEN, SI8>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, int(kLdsLimit));
    if (e != hipSuccess) return e;
    raised.fetch_or(bit, std::memory_order_release);
  }
  hipLaunchKernelGGL((attend_kernel<T, D, RP, LOGITS, TAB, GEN, SI8>), grid, dim3(NT), lds, s, a);
  return hipGetLastError();
}

}  // namespace

template <typename T, int D, int RP>
hipError_t launch_attend_rp(const AttendArgs& a, int batch, bool logits, hipStream_t s) {
  const dim3 grid((unsigned)((a.n_q + BQ - 1) / BQ * a.n_split), (unsigned)a.heads, (unsigned)batch);
  const bool tab = a.tables_in_lds != 0;
  const size_t lds = attend_lds_bytes_t<T, D>(a.rank, a.n_centroids, tab);
  if (lds > kLdsLimit) return hipErrorInvalidValue;
  const bool si8 = a.L.i8 != 0;
  if (logits) {
    if (si8)
      return tab ? launch_k<T, D, RP, true, true, false, true>(a, grid, lds, s)
                 : launch_k<T, D, RP, true, false, false, true>(a, grid, lds, s);
    return tab ? launch_k<T, D, RP, true, true>(a, grid, lds, s) : launch_k<T, D, RP, true, false>(a, grid, lds, s);
  }
  // the general instance: an active chunk, calibration epochs, or sparse PSAC rows
  if (a.n_act > 0 || a.n_epochs > 1 || a.L.sparse) {
    if (si8)
      return tab ? launch_k<T, D, RP, false, true, true, true>(a, grid, lds, s)
                 : launch_k<T, D, RP, false, false, true, true>(a, grid, lds, s);
    return tab ? launch_k<T, D, RP, false, true, true>(a, grid, lds, s)
               : launch_k<T, D, RP, false, false, true>(a, grid, lds, s);
  }
  if (si8)
    return tab ? launch_k<T, D, RP, false, true, false, true>(a, grid, lds, s)
               : launch_k<T, D, RP, false, false, false, true>(a, grid, lds, s);
  return tab ? launch_k<T, D, RP, false, true>(a, grid, lds, s) : launch_k<T, D, RP, false, false>(a, grid, lds, s);
}

template hipError_t launch_attend_rp<QWM_ATTEND_T, QWM_ATTEND_D, QWM_ATTEND_RP>(const AttendArgs&, int, bool,
                                                                                hipStream_t);

}  // namespace qwm
