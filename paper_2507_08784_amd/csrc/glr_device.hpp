// Device building blocks for the gfx950 GreedyLore kernels: MFMA wrappers,
// an LDS-staged fp32 MFMA tile engine with pluggable operand loaders,
// Philox4x32-10 + Box-Muller, and an LDS bitonic sort.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace glr {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4v __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;   // every tiled kernel runs 4 wave64s

// streaming (non-temporal) 16-byte load
__device__ __forceinline__ float4 load_nt4(const float* p) {
  const f32x4v v = __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(p));
  return make_float4(v[0], v[1], v[2], v[3]);
}

// Raw buffer access to one fp32 array of at most 2^32 - 1 bytes: a uniform
// 128-bit descriptor (base, size; no stride) plus a 32-bit byte offset per
// lane.  Offsets at or beyond the size read 0 and drop the store, so a lane
// outside the array passes kBufNone.
typedef __amdgpu_buffer_rsrc_t BufRsrc;
constexpr uint32_t kBufNone = 0xFFFFFFFFu;
// the same for a 16-byte access to an array below 2^31 bytes (no dword of
// it wraps around to a small offset)
constexpr uint32_t kBufNone4 = 0x80000000u;
__device__ __forceinline__ BufRsrc buf_rsrc(const float* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float buf_ld(BufRsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}
__device__ __forceinline__ void buf_st(BufRsrc r, uint32_t off, float x) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, x), r, (int)off, 0, 0);
}

// Storage of the gradients and error buffers: fp32, or bfloat16 (the upper
// half of a binary32) with GLR_STORE_BF16.  A bf16 element widens exactly;
// a store rounds to nearest even (v_cvt_pk_bf16_f32).
typedef uint16_t bf16_t;
__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }
// the value a store of x into ST memory keeps
template <class ST>
__device__ __forceinline__ float stored(float x) {
  if constexpr (sizeof(ST) == 2) return bf16_to_f32(f32_to_bf16(x));
  else return x;
}
__device__ __forceinline__ float ld_e(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_e(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
// elements i .. i + 3 (p + i aligned to four elements)
__device__ __forceinline__ float4 ld_e4(const float* p, int64_t i) {
  return *reinterpret_cast<const float4*>(p + i);
}
__device__ __forceinline__ float4 ld_e4(const bf16_t* p, int64_t i) {
  const uint2 u = *reinterpret_cast<const uint2*>(p + i);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xFFFF0000u));
}
// four elements as loaded (fp32: a float4, bf16: two dwords), widened only
// where the value is used, so that a run of loads is not interrupted by a
// wait for each one
template <class ST>
struct Raw4 {
  float4 v;
};
template <>
struct Raw4<bf16_t> {
  uint2 v;
};
__device__ __forceinline__ Raw4<float> ld_raw4(const float* p, int64_t i) {
  return {*reinterpret_cast<const float4*>(p + i)};
}
__device__ __forceinline__ Raw4<bf16_t> ld_raw4(const bf16_t* p, int64_t i) {
  return {*reinterpret_cast<const uint2*>(p + i)};
}
__device__ __forceinline__ float4 widen4(const Raw4<float>& x) { return x.v; }
__device__ __forceinline__ float4 widen4(const Raw4<bf16_t>& x) {
  return make_float4(__uint_as_float(x.v.x << 16), __uint_as_float(x.v.x & 0xFFFF0000u),
                     __uint_as_float(x.v.y << 16), __uint_as_float(x.v.y & 0xFFFF0000u));
}
template <class ST>
__device__ __forceinline__ Raw4<ST> raw4_zero() {
  Raw4<ST> z;
  if constexpr (sizeof(ST) == 2) z.v = make_uint2(0u, 0u);
  else z.v = make_float4(0.f, 0.f, 0.f, 0.f);
  return z;
}
// the same, streaming (non-temporal)
__device__ __forceinline__ float4 ld_nt_e4(const float* p, int64_t i) { return load_nt4(p + i); }
__device__ __forceinline__ float4 ld_nt_e4(const bf16_t* p, int64_t i) {
  typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
  const u32x2v u = __builtin_nontemporal_load(reinterpret_cast<const u32x2v*>(p + i));
  return make_float4(__uint_as_float(u[0] << 16), __uint_as_float(u[0] & 0xFFFF0000u), __uint_as_float(u[1] << 16),
                     __uint_as_float(u[1] & 0xFFFF0000u));
}
// buffer access to an ST array of `count` elements by the byte offset `off4`
// the element would have in an fp32 array (kBufNone >> 1 still lies beyond
// any bf16 array: count * 2 < 2^31)
template <class ST>
__device__ __forceinline__ BufRsrc buf_rsrc_s(const ST* p, int64_t count) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<ST*>(p), (short)0, (int)(count * (int64_t)sizeof(ST)),
                                           0x00020000);
}
template <class ST>
__device__ __forceinline__ float buf_lde(BufRsrc r, uint32_t off4) {
  if constexpr (sizeof(ST) == 2)
    return bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(r, (int)(off4 >> 1), 0, 0));
  else
    return buf_ld(r, off4);
}
template <class ST>
__device__ __forceinline__ void buf_ste(BufRsrc r, uint32_t off4, float x) {
  if constexpr (sizeof(ST) == 2)
    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(x), r, (int)(off4 >> 1), 0, 0);
  else
    buf_st(r, off4, x);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

// v_mfma_f32_32x32x2_f32:  A 32x2, B 2x32, C 32x32.
//   A[i][k] from lane i + 32k; B[k][j] from lane j + 32k;
//   C[i][j] in lane j + 32*((i/4)%2), register (i%4) + 4*(i/8).
__device__ __forceinline__ f32x16 mfma32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ int mfma32_row(int v, int lane) {
  return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

// v_mfma_f32_32x32x16_bf16:  A 32x16, B 16x32 (bf16), C 32x32 (fp32, laid out
// as for mfma32).  A[i][k] from lane i + 32 (k / 8), element k % 8; B[k][j]
// from lane j + 32 (k / 8), element k % 8.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ f32x16 mfma32_bf16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// v_mfma_f64_16x16x4_f64:  A 16x4, B 4x16, C 16x16 (fp64).
//   A[i][k] from lane i + 16k; B[k][j] from lane j + 16k;
//   C[i][j] in lane j + 16*(i%4), register i/4.
__device__ __forceinline__ f64x4 mfma64(double a, double b, f64x4 c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Operand loaders.  A loader stages a BK x R slice of one GEMM operand into
// LDS in k-major order, s[k * P + r], where r runs over the operand's M (for
// A) or N (for B) dimension.  fetch() issues the global loads into registers,
// put() writes them to LDS, so that the next slice loads while the current
// one feeds the MFMAs.
// ---------------------------------------------------------------------------

// LDS column swizzle of a k-major slice: element (k, r) sits at column
// r ^ lds_swz(k).  It flips bits 2-3 of r only, so the 32 columns one MFMA
// operand read covers stay a permutation of one aligned 32-column block
// (conflict-free reads).
__device__ __forceinline__ constexpr int lds_swz(int k) { return 4 * ((k >> 3) & 3); }

// Element (r, k) at base[row(r) * ld + k] (+ base2[...] when fused): the
// operand is contiguous along k.  Optional row gather through `rows`.  ST is
// the element type in memory (fp32, or bf16 widened as it loads).
// The transposing LDS store puts eight rows x eight float4 k-groups of a
// half-wave in one LDS row pair; with the (R + 4)-float row pitch alone
// those 32 stores meet in 8 banks, and the swizzle spreads them over 32.
// VEC: the caller has checked on the host that `vec` holds (then only the
// float4 path is compiled, and its loads are widened and added in put(), so
// that a fetch issues all its loads before any wait).
template <int R, int BK, bool FUSED, bool GATHER, class ST = float, bool VEC = false>
struct LoadK {
  static constexpr bool kSwz = true;
  static_assert(R % 16 == 0, "swizzle stays inside the slice");
  static constexpr int KQ = BK / 4;                 // float4s per row slice
  static constexpr int NV = (R * KQ + kThreads - 1) / kThreads;
  static constexpr uintptr_t kAl = 4 * sizeof(ST) - 1;   // alignment of four elements
  const ST* base;
  const ST* base2;
  int64_t ld;
  int nrows, K;
  bool vec;
  int64_t roff[NV];
  int rl[NV], kq[NV];
  float4 v[VEC ? 1 : NV];
  Raw4<ST> ra[VEC ? NV : 1], rb[VEC && FUSED ? NV : 1];   // VEC: the loads from base and base2

  __device__ LoadK(const ST* b, const ST* b2, int64_t ld_, int row0, int nrows_, int K_,
                   const int* rows) : base(b), base2(b2), ld(ld_), nrows(nrows_), K(K_) {
    vec = ((ld & 3) == 0) && ((K & 3) == 0) && ((reinterpret_cast<uintptr_t>(b) & kAl) == 0) &&
          (!FUSED || ((reinterpret_cast<uintptr_t>(b2) & kAl) == 0));
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int idx = threadIdx.x + kThreads * i;
      rl[i] = idx / KQ;
      kq[i] = idx % KQ;
      int gr = row0 + rl[i];
      bool ok = (rl[i] < R) && (gr < nrows);
      if (!ok) { roff[i] = -1; continue; }
      int64_t pr = GATHER ? (int64_t)rows[gr] : (int64_t)gr;
      roff[i] = pr * ld;
    }
  }
  __device__ __forceinline__ float ld1(int64_t off) const {
    float x = ld_e(base, off);
    if (FUSED) x += ld_e(base2, off);
    return x;
  }
  // The float4 and the element-wise paths are separate loops under the
  // wave-uniform `vec`: inside one loop the compiler merged the loads of the
  // two paths into shared registers and then waited for every load in
  // flight before issuing the next one.
  __device__ __forceinline__ void fetch(int k0) {
    if constexpr (VEC) fetch_raw(k0);
    else fetch_rt(k0);
  }
  __device__ __forceinline__ void fetch_raw(int k0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = k0 + 4 * kq[i];
      ra[i] = raw4_zero<ST>();
      if (FUSED) rb[FUSED ? i : 0] = raw4_zero<ST>();
      if (roff[i] >= 0 && k < K) {
        ra[i] = ld_raw4(base, roff[i] + k);
        if (FUSED) rb[FUSED ? i : 0] = ld_raw4(base2, roff[i] + k);
      }
    }
  }
  __device__ __forceinline__ void fetch_rt(int k0) {
    if (vec) {
      // K is a multiple of 4 here, and so is k: k < K covers k + 3
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int k = k0 + 4 * kq[i];
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (roff[i] >= 0 && k < K) {
          x = ld_e4(base, roff[i] + k);
          if (FUSED) {
            const float4 y = ld_e4(base2, roff[i] + k);
            x.x += y.x; x.y += y.y; x.z += y.z; x.w += y.w;
          }
        }
        v[i] = x;
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int k = k0 + 4 * kq[i];
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (roff[i] >= 0) {
        int64_t off = roff[i] + k;
        if (k + 0 < K) x.x = ld1(off + 0);
        if (k + 1 < K) x.y = ld1(off + 1);
        if (k + 2 < K) x.z = ld1(off + 2);
        if (k + 3 < K) x.w = ld1(off + 3);
      }
      v[i] = x;
    }
  }
  __device__ __forceinline__ float4 value(int i) const {
    if constexpr (VEC) {
      float4 x = widen4(ra[i]);
      if (FUSED) {
        const float4 y = widen4(rb[FUSED ? i : 0]);
        x.x += y.x; x.y += y.y; x.z += y.z; x.w += y.w;
      }
      return x;
    } else {
      return v[i];
    }
  }
  template <int P>
  __device__ __forceinline__ void put(float* s) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (rl[i] >= R) continue;
      const int k = 4 * kq[i], c = rl[i] ^ lds_swz(k);   // k .. k+3 share the swizzle
      const float4 x = value(i);
      s[(k + 0) * P + c] = x.x;
      s[(k + 1) * P + c] = x.y;
      s[(k + 2) * P + c] = x.z;
      s[(k + 3) * P + c] = x.w;
    }
  }
};

// Element (r, k) at base[krow(k) * ld + r] (+ base2): contiguous along r;
// krow(k) = rows[k] when GATHER, else k.  ST and VEC as for LoadK.
template <int R, int BK, bool FUSED, bool GATHER = false, class ST = float, bool VEC = false>
struct LoadR {
  static constexpr bool kSwz = false;
  static constexpr int RQ = R / 4;
  static constexpr int NV = (BK * RQ + kThreads - 1) / kThreads;
  static constexpr uintptr_t kAl = 4 * sizeof(ST) - 1;
  const ST* base;
  const ST* base2;
  const int* rows;
  int64_t ld;
  int r0, nr, K;
  bool vec;
  int kl[NV], rq[NV];
  float4 v[VEC ? 1 : NV];
  Raw4<ST> ra[VEC ? NV : 1], rb[VEC && FUSED ? NV : 1];   // VEC: the loads from base and base2

  __device__ LoadR(const ST* b, const ST* b2, int64_t ld_, int r0_, int nr_, int K_,
                   const int* rows_ = nullptr)
      : base(b), base2(b2), rows(rows_), ld(ld_), r0(r0_), nr(nr_), K(K_) {
    vec = ((ld & 3) == 0) && ((r0 & 3) == 0) && ((nr & 3) == 0) && ((reinterpret_cast<uintptr_t>(b) & kAl) == 0) &&
          (!FUSED || ((reinterpret_cast<uintptr_t>(b2) & kAl) == 0));
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int idx = threadIdx.x + kThreads * i;
      kl[i] = idx / RQ;
      rq[i] = idx % RQ;
    }
  }
  __device__ __forceinline__ float ld1(int64_t off) const {
    float x = ld_e(base, off);
    if (FUSED) x += ld_e(base2, off);
    return x;
  }
  // float4 and element-wise paths as separate loops under the wave-uniform
  // `vec` (see LoadK::fetch)
  __device__ __forceinline__ void fetch(int k0) {
    if constexpr (VEC) fetch_raw(k0);
    else fetch_rt(k0);
  }
  // the gathered row indices first, so that one wait covers them all
  // (unconditional loads at clamped k, the data loads being masked: a load
  // under a branch is widened inside the branch, which waits for it)
  __device__ __forceinline__ void row_indices(int k0, int (&kr)[NV]) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = k0 + kl[i];
      kr[i] = k;
      if (GATHER && K > 0) kr[i] = rows[k < K ? k : K - 1];
    }
  }
  __device__ __forceinline__ void fetch_raw(int k0) {
    int kr[NV];
    row_indices(k0, kr);
    // nr and r are multiples of 4 here: r < nr covers r + 3
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = k0 + kl[i], r = r0 + 4 * rq[i];
      ra[i] = raw4_zero<ST>();
      if (FUSED) rb[FUSED ? i : 0] = raw4_zero<ST>();
      if (kl[i] < BK && k < K && r < nr) {
        ra[i] = ld_raw4(base, (int64_t)kr[i] * ld + r);
        if (FUSED) rb[FUSED ? i : 0] = ld_raw4(base2, (int64_t)kr[i] * ld + r);
      }
    }
  }
  __device__ __forceinline__ void fetch_rt(int k0) {
    if (vec) {
      int kr[NV];
      row_indices(k0, kr);
      // nr and r are multiples of 4 here: r < nr covers r + 3
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int k = k0 + kl[i], r = r0 + 4 * rq[i];
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
        if (kl[i] < BK && k < K && r < nr) {
          x = ld_e4(base, (int64_t)kr[i] * ld + r);
          if (FUSED) {
            const float4 y = ld_e4(base2, (int64_t)kr[i] * ld + r);
            x.x += y.x; x.y += y.y; x.z += y.z; x.w += y.w;
          }
        }
        v[i] = x;
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int k = k0 + kl[i];
      int r = r0 + 4 * rq[i];
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (kl[i] < BK && k < K) {
        const int64_t kr = GATHER ? (int64_t)rows[k] : (int64_t)k;
        int64_t off = kr * ld + r;
        if (r + 0 < nr) x.x = ld1(off + 0);
        if (r + 1 < nr) x.y = ld1(off + 1);
        if (r + 2 < nr) x.z = ld1(off + 2);
        if (r + 3 < nr) x.w = ld1(off + 3);
      }
      v[i] = x;
    }
  }
  __device__ __forceinline__ float4 value(int i) const {
    if constexpr (VEC) {
      float4 x = widen4(ra[i]);
      if (FUSED) {
        const float4 y = widen4(rb[FUSED ? i : 0]);
        x.x += y.x; x.y += y.y; x.z += y.z; x.w += y.w;
      }
      return x;
    } else {
      return v[i];
    }
  }
  template <int P>
  __device__ __forceinline__ void put(float* s) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (kl[i] >= BK) continue;
      *reinterpret_cast<float4*>(s + kl[i] * P + 4 * rq[i]) = value(i);
    }
  }
};

// LoadR's float4 case on a buffer descriptor: element (r, k) of the fp32
// operand at byte off0 + 4 (krow(k) ld + r) of the descriptor's array (below
// 2^31 bytes; ld, r0 and nr multiples of 4).  Every load is issued
// unconditionally, an element outside the slice or the operand reading 0
// through an offset past the array, so a fetch is one run of loads with no
// branch between them (under branches, the compiler's waits for loads it
// cannot track made each load wait for the previous ones).
template <int R, int BK, bool GATHER>
struct LoadRB {
  static constexpr bool kSwz = false;
  static constexpr int RQ = R / 4;
  static constexpr int NV = (BK * RQ + kThreads - 1) / kThreads;
  BufRsrc rs;
  uint32_t off0;
  const int* rows;
  int ld, r0, nr, K;
  int kl[NV], rq[NV];
  float4 v[NV];

  __device__ LoadRB(BufRsrc rs_, uint32_t off0_, int ld_, int r0_, int nr_, int K_, const int* rows_ = nullptr)
      : rs(rs_), off0(off0_), rows(rows_), ld(ld_), r0(r0_), nr(nr_), K(K_) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + kThreads * i;
      kl[i] = idx / RQ;
      rq[i] = idx % RQ;
    }
  }
  __device__ __forceinline__ void fetch(int k0) {
    int kr[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = k0 + kl[i];
      kr[i] = k;
      if (GATHER && K > 0) kr[i] = rows[k < K ? k : K - 1];   // clamped: the data load below is dropped
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = k0 + kl[i], r = r0 + 4 * rq[i];
      const bool ok = kl[i] < BK && k < K && r < nr;
      const uint32_t off = ok ? off0 + 4u * (uint32_t)(kr[i] * ld + r) : kBufNone4;
      const auto x = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, 0, 0);
      v[i] = make_float4(__uint_as_float(x[0]), __uint_as_float(x[1]), __uint_as_float(x[2]), __uint_as_float(x[3]));
    }
  }
  template <int P>
  __device__ __forceinline__ void put(float* s) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (kl[i] >= BK) continue;
      *reinterpret_cast<float4*>(s + kl[i] * P + 4 * rq[i]) = v[i];
    }
  }
};

// ---------------------------------------------------------------------------
// MFMA tile engine: C[BM x BN] = A[BM x K] B[K x BN] in fp32 with
// v_mfma_f32_32x32x2_f32.  4 waves in a WM x WN grid; each wave owns a
// (BM/WM) x (BN/WN) sub-tile of TM x TN MFMA blocks.  LDS holds one k-major
// slice per operand; the next slice is prefetched into registers while the
// current one feeds the MFMAs.
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN>
struct MfmaTile {
  static constexpr int BK = 32;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static constexpr int PA = BM + 4, PB = BN + 4;
  static constexpr int SA = BK * PA, SB = BK * PB;
  static constexpr int LDS_FLOATS = SA + SB;
  static_assert(WM * WN == 4, "4 waves");
  static_assert(TM >= 1 && TN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "32x32 blocks");

  f32x16 acc[TM][TN];
  int wm, wn, lane;

  __device__ MfmaTile() {
    lane = lane_id();
    wm = wave_id() / WN;
    wn = wave_id() % WN;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  }

  // tile-relative row / column of accumulator element (tm, tn, v)
  __device__ __forceinline__ int row(int tm, int v) const {
    return wm * WTM + tm * 32 + mfma32_row(v, lane);
  }
  __device__ __forceinline__ int col(int tn) const { return wn * WTN + tn * 32 + (lane & 31); }

  // SWA / SWB: the operand's slice is stored with the lds_swz column swizzle
  template <bool SWA, bool SWB>
  __device__ __forceinline__ void compute(const float* As, const float* Bs) {
    const int kh = lane >> 5, l32 = lane & 31;
#pragma unroll
    for (int kk = 0; kk < BK / 2; ++kk) {
      // rows 2 kk and 2 kk + 1 share one swizzle
      const int ca = SWA ? (l32 ^ lds_swz(2 * kk)) : l32;
      const int cb = SWB ? (l32 ^ lds_swz(2 * kk)) : l32;
      float a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) a[i] = As[(2 * kk + kh) * PA + wm * WTM + i * 32 + ca];
#pragma unroll
      for (int j = 0; j < TN; ++j) b[j] = Bs[(2 * kk + kh) * PB + wn * WTN + j * 32 + cb];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
    }
  }

  // the same product with both operands rounded to bf16 (to nearest even) as
  // they leave LDS, fp32 accumulation: two bf16 MFMAs of depth 16 per slice
  template <bool SWA, bool SWB>
  __device__ __forceinline__ void compute_bf16(const float* As, const float* Bs) {
    const int kh = lane >> 5, l32 = lane & 31;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      // rows 16 ks + 8 kh .. + 7 share one swizzle
      const int ca = SWA ? (l32 ^ lds_swz(16 * ks + 8 * kh)) : l32;
      const int cb = SWB ? (l32 ^ lds_swz(16 * ks + 8 * kh)) : l32;
      bf16x8 a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) a[i][e] = (__bf16)As[(16 * ks + 8 * kh + e) * PA + wm * WTM + i * 32 + ca];
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) b[j][e] = (__bf16)Bs[(16 * ks + 8 * kh + e) * PB + wn * WTN + j * 32 + cb];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32_bf16(a[i], b[j], acc[i][j]);
    }
  }

  // acc += A B over K (BF16: with both operands rounded to bf16).  With `dacc`,
  // the fp32 accumulators are added into fp64 ones after every 16 BK slices
  // and cleared, so that rounding grows with that length only (dacc holds the
  // result then; acc is zero).
  template <bool BF16 = false, class LA, class LB>
  __device__ void run(LA& la, LB& lb, int K, float* smem, double (*dacc)[TN][16] = nullptr) {
    float* As = smem;
    float* Bs = smem + SA;
    const int nk = (K + BK - 1) / BK;
    if (nk == 0) return;
    la.fetch(0);
    lb.fetch(0);
    la.template put<PA>(As);
    lb.template put<PB>(Bs);
    __syncthreads();
    for (int kb = 0; kb < nk; ++kb) {
      const bool more = kb + 1 < nk;
      if (more) {
        la.fetch((kb + 1) * BK);
        lb.fetch((kb + 1) * BK);
      }
      if constexpr (BF16) compute_bf16<LA::kSwz, LB::kSwz>(As, Bs);
      else compute<LA::kSwz, LB::kSwz>(As, Bs);
      if (dacc && ((kb & 15) == 15 || !more)) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              dacc[i][j][v] += (double)acc[i][j][v];
              acc[i][j][v] = 0.f;
            }
      }
      __syncthreads();
      if (more) {
        la.template put<PA>(As);
        lb.template put<PB>(Bs);
        __syncthreads();
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11) and Box-Muller normals.
// Element b of v_j (matrix l, step t) comes from counter (b/4, j, l, t) under
// key (seed lo, seed hi); words (x0,x1) give b = 4c, 4c+1 and (x2,x3) give
// 4c+2, 4c+3; u(x) = (x >> 9) 2^-23 + 2^-24.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void philox4x32_10(uint32_t& c0, uint32_t& c1, uint32_t& c2, uint32_t& c3,
                                              uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    const uint32_t a = c0, b = c2;
    const uint32_t hi_a = __umulhi(0xD2511F53u, a), lo_a = 0xD2511F53u * a;
    const uint32_t hi_b = __umulhi(0xCD9E8D57u, b), lo_b = 0xCD9E8D57u * b;
    c0 = hi_b ^ c1 ^ k0;
    c1 = lo_b;
    c2 = hi_a ^ c3 ^ k1;
    c3 = lo_a;
  }
}

__device__ __forceinline__ float uniform01(uint32_t x) {
  return (float)(x >> 9) * 0x1p-23f + 0x1p-24f;
}

__device__ __forceinline__ void box_muller(uint32_t xa, uint32_t xb, float& z0, float& z1) {
  const float rho = sqrtf(-2.0f * logf(uniform01(xa)));
  float s, c;
  sincospif(2.0f * uniform01(xb), &s, &c);
  z0 = rho * c;
  z1 = rho * s;
}

// the four normals v_j[4c .. 4c+3]
__device__ __forceinline__ void normals4(uint32_t c, uint32_t j, uint32_t mat, uint32_t t,
                                         uint32_t k0, uint32_t k1, float z[4]) {
  uint32_t x0 = c, x1 = j, x2 = mat, x3 = t;
  philox4x32_10(x0, x1, x2, x3, k0, k1);
  box_muller(x0, x1, z[0], z[1]);
  box_muller(x2, x3, z[2], z[3]);
}

// ---------------------------------------------------------------------------
// reductions and sorting
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ double wave_max(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o, 64));
  return x;
}

// order-preserving map of a float to uint32 (ascending)
__device__ __forceinline__ uint32_t float_order(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ascending bitonic sort of n (power of two) 64-bit keys in LDS, whole block
__device__ inline void bitonic_sort(uint64_t* s, int n) {
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < n; i += blockDim.x) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = s[i], b = s[ixj];
          const bool up = (i & k) == 0;
          if ((a > b) == up) { s[i] = b; s[ixj] = a; }
        }
      }
      __syncthreads();
    }
  }
}

}  // namespace glr
