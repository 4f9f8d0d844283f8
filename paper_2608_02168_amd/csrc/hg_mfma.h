// MFMA building blocks for gfx950 (fp32 path: v_mfma_f32_16x16x4_f32).
//
// Lane layouts (64-lane wave, g = lane / 16, c = lane % 16):
//   A operand (16 x 4):  lane holds A[c][g]
//   B operand (4 x 16):  lane holds B[g][c]
//   C/D (16 x 16):       lane holds D[4 g + v][c] in accumulator register v
//
// Two kernels are built on it:
//   gemm_rows   C[rows] = epi(A[rows] . op(W))   with W (d x d) staged in LDS,
//               rows gathered through a row map; a 16-wide K block is split
//               so each lane reads 4 consecutive A elements (one float4),
//               matched by the same K permutation of W inside LDS;
//   gemm_tn     partial[chunk] = A[rows]^T B[rows] over a chunk of rows,
//               a deterministic split-K for weight gradients and Gram matrices.
#pragma once

#include <type_traits>

#include "hg_internal.h"

namespace hg {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t bf16_t;  // bfloat16 storage

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bfloat16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack2bf(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

// Element types of feature rows: 16-byte chunks hold EL elements.
template <class T>
struct Elt;
template <>
struct Elt<float> {
  static constexpr int EL = 4;
  typedef float vf __attribute__((ext_vector_type(4)));
  typedef double vd __attribute__((ext_vector_type(4)));
  __device__ static __forceinline__ vf loadv(const float* p) { return *reinterpret_cast<const vf*>(p); }
  __device__ static __forceinline__ void load(const float* p, float (&v)[4]) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(p);
    v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3];
  }
  __device__ static __forceinline__ void store(float* p, const float (&v)[4]) {
    *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
  }
  __device__ static __forceinline__ float get(const float* p) { return *p; }
  __device__ static __forceinline__ f32x4 load4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  // four elements as loaded (issue) and as used (after the data arrived)
  typedef f32x4 raw4_t;
  __device__ static __forceinline__ raw4_t raw4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  __device__ static __forceinline__ f32x4 cook4(raw4_t r) { return r; }
  // one 16-byte chunk (EL elements) as loaded; element k is unpacked where it
  // is used, so a gather keeps 4 registers per row in flight
  typedef f32x4 rawv_t;
  __device__ static __forceinline__ rawv_t rawv(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
  __device__ static __forceinline__ rawv_t rawv_zero() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
  __device__ static __forceinline__ float rawv_get(const rawv_t& x, int k) { return x[k]; }
};
template <>
struct Elt<bf16_t> {
  static constexpr int EL = 8;
  typedef float vf __attribute__((ext_vector_type(8)));
  typedef double vd __attribute__((ext_vector_type(8)));
  __device__ static __forceinline__ vf loadv(const bf16_t* p) {
    const uint4 x = *reinterpret_cast<const uint4*>(p);
    vf v;
    v[0] = __uint_as_float(x.x << 16); v[1] = __uint_as_float(x.x & 0xFFFF0000u);
    v[2] = __uint_as_float(x.y << 16); v[3] = __uint_as_float(x.y & 0xFFFF0000u);
    v[4] = __uint_as_float(x.z << 16); v[5] = __uint_as_float(x.z & 0xFFFF0000u);
    v[6] = __uint_as_float(x.w << 16); v[7] = __uint_as_float(x.w & 0xFFFF0000u);
    return v;
  }
  __device__ static __forceinline__ void load(const bf16_t* p, float (&v)[8]) {
    const uint4 x = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[2 * q] = __uint_as_float(w[q] << 16);
      v[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
    }
  }
  __device__ static __forceinline__ void store(bf16_t* p, const float (&v)[8]) {
    uint4 x;
    x.x = pack2bf(v[0], v[1]);
    x.y = pack2bf(v[2], v[3]);
    x.z = pack2bf(v[4], v[5]);
    x.w = pack2bf(v[6], v[7]);
    *reinterpret_cast<uint4*>(p) = x;
  }
  __device__ static __forceinline__ float get(const bf16_t* p) { return bf2f(*p); }
  __device__ static __forceinline__ f32x4 load4(const bf16_t* p) {
    const uint2 x = *reinterpret_cast<const uint2*>(p);
    return f32x4{__uint_as_float(x.x << 16), __uint_as_float(x.x & 0xFFFF0000u),
                 __uint_as_float(x.y << 16), __uint_as_float(x.y & 0xFFFF0000u)};
  }
  typedef uint2 raw4_t;
  __device__ static __forceinline__ raw4_t raw4(const bf16_t* p) { return *reinterpret_cast<const uint2*>(p); }
  __device__ static __forceinline__ f32x4 cook4(raw4_t x) {
    return f32x4{__uint_as_float(x.x << 16), __uint_as_float(x.x & 0xFFFF0000u),
                 __uint_as_float(x.y << 16), __uint_as_float(x.y & 0xFFFF0000u)};
  }
  typedef u32x4 rawv_t;
  __device__ static __forceinline__ rawv_t rawv(const bf16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
  __device__ static __forceinline__ rawv_t rawv_zero() { return u32x4{0u, 0u, 0u, 0u}; }
  // element 2q is the low half of word q, element 2q + 1 the high half
  __device__ static __forceinline__ float rawv_get(const rawv_t& x, int k) {
    return (k & 1) ? __uint_as_float(x[k >> 1] & 0xFFFF0000u) : __uint_as_float(x[k >> 1] << 16);
  }
};

__device__ __forceinline__ f32x4 mfma_bf16(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                 c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---- split-fp16 products ------------------------------------------------------
// A float32 product x w is formed on the fp16 MFMA from two fp16 parts of each
// factor: with 2^ex the power of two that brings the largest |x| of a scaled
// group into [2^14, 2^15),  xh = fp16(x 2^ex)  and  xl = fp16(x 2^ex - xh),
// likewise for w, and
//   x w ~= 2^-(ex+ew) (xh wh + xh wl + xl wh).
// The three fp16 MFMAs accumulate into one float32 accumulator (fp16 products
// are exact in float32) and do the work of one K=32 block at 3/16 of the cost
// of the float32 MFMA.  The omitted xl wl term and the two conversions leave
// a relative error of about 2^-21 of the group's largest magnitude, near
// float32 rounding.  Scaling by powers of two is exact; the range [2^14, 2^15)
// keeps every part below the fp16 maximum, and a low part falls into the fp16
// subnormal range only below 2^-28 of the group's largest magnitude.
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x4 mfma_f16(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                0, 0, 0);
}

// Biased float32 exponent of the largest magnitude m of a group, clamped so
// that both 2^(14 - e) and 2^(e - 14) (e the unbiased exponent) are normal.
__device__ __forceinline__ uint32_t split_exp(float m) {
  uint32_t eb = (__float_as_uint(m) >> 23) & 0xFFu;
  return eb < 15u ? 15u : (eb > 254u ? 254u : eb);
}
// 2^(14 - e): multiplies the group into [2^14, 2^15)
__device__ __forceinline__ float split_scale(uint32_t eb) { return __uint_as_float((268u - eb) << 23); }
// 2^(e - 14): undoes split_scale
__device__ __forceinline__ float split_unscale(uint32_t eb) { return __uint_as_float((eb - 14u) << 23); }

// Eight scaled values -> fp16 high parts and fp16 remainders.
__device__ __forceinline__ void split8(const float (&v)[8], uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const auto hp = __builtin_amdgcn_cvt_pkrtz(v[2 * q], v[2 * q + 1]);
    const float r0 = v[2 * q] - (float)hp[0];
    const float r1 = v[2 * q + 1] - (float)hp[1];
    h[q] = __builtin_bit_cast(uint32_t, hp);
    l[q] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(r0, r1));
  }
  hi = uint4{h[0], h[1], h[2], h[3]};
  lo = uint4{l[0], l[1], l[2], l[3]};
}

// acc unscaled by the two factors' scales one after the other (their product
// alone could leave the normal range)
__device__ __forceinline__ f32x4 split_unscale4(f32x4 acc, float ux, float uw) {
  f32x4 r;
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = (acc[v] * ux) * uw;
  return r;
}

__device__ __forceinline__ int lane64() { return threadIdx.x & 63; }

// Row map: row(i) = (list ? list[i] : first + i) * mul + add.
struct RowMap {
  const int32_t* list;
  int64_t first;
  int32_t mul;
  int32_t add;
  __device__ __forceinline__ int64_t operator()(int64_t i) const {
    const int64_t b = list ? (int64_t)list[i] : first + i;
    return b * mul + add;
  }
  // The same split in two with the list/contiguous choice fixed at compile
  // time: key(i) is the raw list entry (a load whose value is not touched) or
  // i itself; row_of(key) does the arithmetic once the entry has arrived.
  template <bool kList>
  using Key = typename std::conditional<kList, int32_t, int64_t>::type;
  template <bool kList>
  __device__ __forceinline__ Key<kList> key(int64_t i) const {
    if constexpr (kList) {
      return list[i];
    } else {
      return i;
    }
  }
  template <bool kList>
  __device__ __forceinline__ int64_t row_of(Key<kList> k) const {
    if constexpr (kList) {
      return (int64_t)k * mul + add;
    } else {
      return (first + k) * mul + add;
    }
  }
};

inline RowMap rows_contig(int64_t first) { return RowMap{nullptr, first, 1, 0}; }
inline RowMap rows_list(const int32_t* list, int32_t mul = 1, int32_t add = 0) {
  return RowMap{list, 0, mul, add};
}

// ---- A loaders: rowp(i) = address of segment row i; load4 / load1 read
// columns of that row (with an optional per-column transform) ------------------
template <int D, class T = float>
struct LoadRows {
  const T* base;
  RowMap map;
  __device__ __forceinline__ const T* rowp(int64_t i) const { return base + map(i) * D; }
  __device__ __forceinline__ f32x4 load4(const T* p, int c) const { return Elt<T>::load4(p + c); }
  // 8 consecutive columns as bfloat16 (the bf16 MFMA operand)
  __device__ __forceinline__ uint4 load8bf(const T* p, int c) const {
    if constexpr (sizeof(T) == 2) {
      return *reinterpret_cast<const uint4*>(p + c);
    } else {
      const f32x4 x = load4(p, c), y = load4(p, c + 4);
      return uint4{pack2bf(x[0], x[1]), pack2bf(x[2], x[3]), pack2bf(y[0], y[1]), pack2bf(y[2], y[3])};
    }
  }
  __device__ __forceinline__ float load1(const T* p, int c) const { return Elt<T>::get(p + c); }
  __device__ __forceinline__ float at(int64_t i, int c) const { return load1(rowp(i), c); }
  // split form for prefetching: base row, raw load, transform at use
  typedef typename Elt<T>::raw4_t Raw;
  struct Prep {};
  __device__ __forceinline__ Raw raw4b(int64_t b, int c) const { return Elt<T>::raw4(base + b * D + c); }
  __device__ __forceinline__ Prep prep(int) const { return Prep{}; }
  __device__ __forceinline__ f32x4 cook4(Raw r, const Prep&) const { return Elt<T>::cook4(r); }
  // whole-row form of the split (lane group g holds columns 16 kb + 4 g)
  struct RowRaw {
    Raw x[D / 16];
  };
  __device__ __forceinline__ void fetch_row(int64_t b, int g, RowRaw& r) const {
#pragma unroll
    for (int kb = 0; kb < D / 16; ++kb) r.x[kb] = raw4b(b, 16 * kb + 4 * g);
  }
  __device__ __forceinline__ void cook_row(const RowRaw& r, int64_t, int, bool, f32x4 (&a)[D / 16]) const {
#pragma unroll
    for (int kb = 0; kb < D / 16; ++kb) a[kb] = Elt<T>::cook4(r.x[kb]);
  }
  // per-K-block form: the row as stored, and the MFMA operand
  __device__ __forceinline__ f32x4 stored4(const RowRaw& r, int kb) const { return Elt<T>::cook4(r.x[kb]); }
  __device__ __forceinline__ f32x4 stored4r(const Raw& r) const { return Elt<T>::cook4(r); }
  __device__ __forceinline__ f32x4 operand4(const RowRaw& r, int kb, int) const { return Elt<T>::cook4(r.x[kb]); }
  static constexpr bool kTee = false;
  static constexpr bool kBoundByStored = false;
  static constexpr bool kHalf = sizeof(T) == 2;
  __device__ __forceinline__ void tee4(int64_t, int, int, f32x4) const {}
};

// (x - mu[c]) * sc[c]: the per-column standardisation of the alignment loss.
template <int D, class T = float>
struct LoadStd {
  const T* base;
  RowMap map;
  const float* mu;
  const float* sc;
  __device__ __forceinline__ const T* rowp(int64_t i) const { return base + map(i) * D; }
  __device__ __forceinline__ uint4 load8bf(const T* p, int c) const {
    const f32x4 x = load4(p, c), y = load4(p, c + 4);
    return uint4{pack2bf(x[0], x[1]), pack2bf(x[2], x[3]), pack2bf(y[0], y[1]), pack2bf(y[2], y[3])};
  }
  __device__ __forceinline__ f32x4 load4(const T* p, int c) const {
    f32x4 x = Elt<T>::load4(p + c);
    f32x4 m = *reinterpret_cast<const f32x4*>(mu + c);
    f32x4 s = *reinterpret_cast<const f32x4*>(sc + c);
    f32x4 r;
    r[0] = (x[0] - m[0]) * s[0];
    r[1] = (x[1] - m[1]) * s[1];
    r[2] = (x[2] - m[2]) * s[2];
    r[3] = (x[3] - m[3]) * s[3];
    return r;
  }
  __device__ __forceinline__ float load1(const T* p, int c) const { return (Elt<T>::get(p + c) - mu[c]) * sc[c]; }
  __device__ __forceinline__ float at(int64_t i, int c) const { return load1(rowp(i), c); }
  typedef typename Elt<T>::raw4_t Raw;
  struct Prep {
    f32x4 m, s;
  };
  __device__ __forceinline__ Raw raw4b(int64_t b, int c) const { return Elt<T>::raw4(base + b * D + c); }
  __device__ __forceinline__ Prep prep(int c) const {
    return Prep{*reinterpret_cast<const f32x4*>(mu + c), *reinterpret_cast<const f32x4*>(sc + c)};
  }
  __device__ __forceinline__ f32x4 cook4(Raw raw, const Prep& q) const {
    const f32x4 x = Elt<T>::cook4(raw);
    f32x4 r;
    r[0] = (x[0] - q.m[0]) * q.s[0];
    r[1] = (x[1] - q.m[1]) * q.s[1];
    r[2] = (x[2] - q.m[2]) * q.s[2];
    r[3] = (x[3] - q.m[3]) * q.s[3];
    return r;
  }
};

// dZ = G * mask read on the fly: the ReLU mask row of G row r holds bit c of
// column c at word r*(D/32) + c/32.
template <int D, class T = float>
struct LoadMasked {
  const T* G;
  const uint32_t* mask;
  RowMap map;
  T* tee;  // if set, loads also store the masked values here (same offsets as G)
  __device__ __forceinline__ const T* rowp(int64_t i) const { return G + map(i) * D; }
  __device__ __forceinline__ uint32_t word(const T* p, int c) const {
    const int64_t r = (p - G) / D;
    return mask[r * (D / 32) + (c >> 5)];
  }
  __device__ __forceinline__ f32x4 load4(const T* p, int c) const {
    f32x4 x = Elt<T>::load4(p + c);
    const uint32_t nib = word(p, c) >> (c & 31);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (!((nib >> q) & 1u)) x[q] = 0.f;
    if (tee) {
      if constexpr (sizeof(T) == 4) {
        *reinterpret_cast<f32x4*>(tee + (p - G) + c) = x;
      } else {
        *reinterpret_cast<uint2*>(tee + (p - G) + c) = uint2{pack2bf(x[0], x[1]), pack2bf(x[2], x[3])};
      }
    }
    return x;
  }
  __device__ __forceinline__ uint4 load8bf(const T* p, int c) const {
    static_assert(sizeof(T) == 2, "load8bf of masked rows is the bfloat16 path");
    uint4 x = *reinterpret_cast<const uint4*>(p + c);
    const uint32_t byte = (word(p, c) >> (c & 31)) & 0xFFu;
    uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = ((byte >> (2 * q)) & 1u) ? 0x0000FFFFu : 0u;
      const uint32_t hi = ((byte >> (2 * q + 1)) & 1u) ? 0xFFFF0000u : 0u;
      w[q] &= (lo | hi);
    }
    x = uint4{w[0], w[1], w[2], w[3]};
    if (tee) *reinterpret_cast<uint4*>(tee + (p - G) + c) = x;
    return x;
  }
  __device__ __forceinline__ float load1(const T* p, int c) const {
    return ((word(p, c) >> (c & 31)) & 1u) ? Elt<T>::get(p + c) : 0.f;
  }
  __device__ __forceinline__ float at(int64_t i, int c) const { return load1(rowp(i), c); }
  // Whole-row split: the row's elements and its D/32 mask words are loaded
  // first; the mask is applied (and the masked values written to tee) when
  // they are used.  Lane group g holds columns 16 kb + 4 g.
  typedef typename Elt<T>::raw4_t Raw;
  struct RowRaw {
    Raw x[D / 16];
    uint32_t m[D / 32];
  };
  __device__ __forceinline__ void fetch_row(int64_t b, int g, RowRaw& r) const {
#pragma unroll
    for (int kb = 0; kb < D / 16; ++kb) r.x[kb] = Elt<T>::raw4(G + b * D + 16 * kb + 4 * g);
    const uint32_t* mw = mask + b * (D / 32);
    if constexpr (D == 64) {
      const uint2 v = *reinterpret_cast<const uint2*>(mw);
      r.m[0] = v.x; r.m[1] = v.y;
    } else {
#pragma unroll
      for (int q = 0; q < D / 128; ++q) {
        const uint4 v = *reinterpret_cast<const uint4*>(mw + 4 * q);
        r.m[4 * q] = v.x; r.m[4 * q + 1] = v.y; r.m[4 * q + 2] = v.z; r.m[4 * q + 3] = v.w;
      }
    }
  }
  __device__ __forceinline__ void cook_row(const RowRaw& r, int64_t b, int g, bool live, f32x4 (&a)[D / 16]) const {
#pragma unroll
    for (int kb = 0; kb < D / 16; ++kb) {
      f32x4 x = Elt<T>::cook4(r.x[kb]);
      const uint32_t nib = r.m[kb >> 1] >> (16 * (kb & 1) + 4 * g);
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = ((nib >> q) & 1u) ? x[q] : 0.f;
      if (tee && live) {
        T* o = tee + b * D + 16 * kb + 4 * g;
        if constexpr (sizeof(T) == 4) {
          *reinterpret_cast<f32x4*>(o) = x;
        } else {
          *reinterpret_cast<uint2*>(o) = uint2{pack2bf(x[0], x[1]), pack2bf(x[2], x[3])};
        }
      }
      a[kb] = x;
    }
  }
  __device__ __forceinline__ f32x4 stored4(const RowRaw& r, int kb) const { return Elt<T>::cook4(r.x[kb]); }
  __device__ __forceinline__ f32x4 stored4r(const Raw& r) const { return Elt<T>::cook4(r); }
  __device__ __forceinline__ f32x4 operand4(const RowRaw& r, int kb, int g) const {
    f32x4 x = Elt<T>::cook4(r.x[kb]);
    const uint32_t nib = r.m[kb >> 1] >> (16 * (kb & 1) + 4 * g);
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = ((nib >> q) & 1u) ? x[q] : 0.f;
    return x;
  }
  static constexpr bool kTee = true;
  // |operand| <= |stored| element by element (the mask only zeroes)
  static constexpr bool kBoundByStored = true;
  static constexpr bool kHalf = sizeof(T) == 2;
  __device__ __forceinline__ void tee4(int64_t b, int kb, int g, f32x4 x) const {
    if (!tee) return;
    T* o = tee + b * D + 16 * kb + 4 * g;
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<f32x4*>(o) = x;
    } else {
      *reinterpret_cast<uint2*>(o) = uint2{pack2bf(x[0], x[1]), pack2bf(x[2], x[3])};
    }
  }
};

// ---- epilogues ------------------------------------------------------------
// The kernel calls row(i) once per output row, then pre(i, ro, c) for every
// element of the tile (all loads), then store(i, ro, c, acc, pre) (all stores):
// the two phases keep loads from waiting behind stores when the addend is the
// output itself (dH += ...).
// kAddendIsA: the addend rows are the A operand's rows as stored (before the
// loader's transform), at the same row index; a kernel holding those rows in
// registers may use them instead of reading the addend again.
template <int D, class T = float, class TA = T, bool kAddendIsA = false>
struct StoreRows {
  static constexpr bool kAddA = kAddendIsA;
  static constexpr bool kMask = false;
  T* out;
  RowMap map;
  const float* bias;  // [D] or null
  const TA* addend;   // rows through the same map, or null (may equal out)
  __device__ __forceinline__ int64_t row(int64_t i) const { return map(i); }
  __device__ __forceinline__ float pre(int64_t, int64_t ro, int c) const {
    float v = bias ? bias[c] : 0.f;
    if (addend) v += Elt<TA>::get(addend + ro * D + c);
    return v;
  }
  __device__ __forceinline__ void store(int64_t, int64_t ro, int c, float acc, float pre) const {
    if constexpr (sizeof(T) == 4) {
      out[ro * D + c] = acc + pre;
    } else {
      out[ro * D + c] = f2bf(acc + pre);
    }
  }
  // four consecutive columns [c, c + 4) of one row
  __device__ __forceinline__ f32x4 pre4(int64_t, int64_t ro, int c) const {
    f32x4 v = bias ? *reinterpret_cast<const f32x4*>(bias + c) : f32x4{0.f, 0.f, 0.f, 0.f};
    if (addend) v += Elt<TA>::load4(addend + ro * D + c);
    return v;
  }
  __device__ __forceinline__ f32x4 bias4(int c) const {
    return bias ? *reinterpret_cast<const f32x4*>(bias + c) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __device__ __forceinline__ void store4(int64_t, int64_t ro, int c, f32x4 acc, f32x4 pre) const {
    const f32x4 r = acc + pre;
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<f32x4*>(out + ro * D + c) = r;
    } else {
      *reinterpret_cast<uint2*>(out + ro * D + c) = uint2{pack2bf(r[0], r[1]), pack2bf(r[2], r[3])};
    }
  }
};

// dH rows of a bfloat16 layer, each written once in bf16: the self pass and
// the relation passes in relation order add into a float32 accumulator, and
// the last pass that reaches a row writes it in bf16 instead.  Relation pass
// r (r = -1: the self pass) is a row's last when the row has no CSC entries
// of a relation after r: csc_ptr[i R + R] == csc_ptr[i R + r + 1].  The self
// pass writes the accumulator of every row some relation pass reaches after
// it, so each relation pass reads an initialised accumulator (its addend).
template <int D, class TA = float, bool kAddendIsA = false>
struct StoreLast {
  static constexpr bool kAddA = kAddendIsA;
  static constexpr bool kMask = false;
  static constexpr bool kRowFlag = true;  // the kernel reads last(ro) once per row, early
  bf16_t* out;          // [rows, D] final bf16 rows
  float* accum;         // [rows, D] float32 accumulator rows
  RowMap map;
  const float* bias;    // [D] or null
  const TA* addend;     // rows through the same map (the accumulator, or the residual), or null
  const int32_t* csc_ptr;
  int32_t n_rel, rel;   // rel = -1 for the self pass
  __device__ __forceinline__ int64_t row(int64_t i) const { return map(i); }
  __device__ __forceinline__ bool last(int64_t ro) const {
    const int32_t* q = csc_ptr + ro * n_rel;
    return q[n_rel] == q[rel + 1];
  }
  __device__ __forceinline__ f32x4 pre4(int64_t, int64_t ro, int c) const {
    f32x4 v = bias ? *reinterpret_cast<const f32x4*>(bias + c) : f32x4{0.f, 0.f, 0.f, 0.f};
    if (addend) v += Elt<TA>::load4(addend + ro * D + c);
    return v;
  }
  __device__ __forceinline__ f32x4 bias4(int c) const {
    return bias ? *reinterpret_cast<const f32x4*>(bias + c) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __device__ __forceinline__ bool flag(int64_t ro) const { return last(ro); }
  __device__ __forceinline__ void store4f(int64_t, int64_t ro, int c, f32x4 acc, f32x4 pre, bool is_last) const {
    const f32x4 r = acc + pre;
    if (is_last) {
      *reinterpret_cast<uint2*>(out + ro * D + c) = uint2{pack2bf(r[0], r[1]), pack2bf(r[2], r[3])};
    } else {
      *reinterpret_cast<f32x4*>(accum + ro * D + c) = r;
    }
  }
};

// Epilogues with kRowFlag take a per-row flag, read once per row before the
// products (flag(ro)), in their stores (store4f).
// loaders whose rows are stored in a 16-bit type (kHalf)
template <class L, class = void>
struct HalfRows : std::false_type {};
template <class L>
struct HalfRows<L, std::void_t<decltype(L::kHalf)>> : std::integral_constant<bool, L::kHalf> {};

template <class E, class = void>
struct EpiRowFlag : std::false_type {};
template <class E>
struct EpiRowFlag<E, std::void_t<decltype(E::kRowFlag)>> : std::integral_constant<bool, E::kRowFlag> {};

// ---- row GEMMs on the split-fp16 MFMA: shared shape ------------------------------
// Block = 8 waves (16 at d = 256) sharing one LDS copy of a column slice of
// op(W); a wave owns 16 rows of a tile; persistent over tiles.  W is D x D;
// the column slice is [DN s, DN s + DN) (DN = D for D <= 128, 128 for
// D = 256; the block index picks s and the tile group, see the kernel).
// Products on the split-fp16 MFMA (split8): each row is scaled by the power
// of two of its largest magnitude, op(W) by that of its own; LDS holds the
// slice in fragment order, uint4 element (kb2*NB + nb)*64 + lane being
// op(W)[k][col0 + 16 nb + lane%16] for the lane's 8 K slots of K block kb2
// (columns 16 (2 kb2) + 4 (lane/16) .. + 3 and the same 16 further on), high
// parts first, then the remainders.
constexpr int kGemmThreads = 512;
template <int D>
struct F32Slice {
  static constexpr int DN = D > 128 ? 128 : D;
};

// ---- gemm_rows on the split-fp16 MFMA ------------------------------------------------
// Row GEMM on the split-fp16 MFMA (v_mfma_f32_16x16x32_f16, three products
// per K block, see split8): tiles of 16 rows per wave, 8 waves per block (16
// without prefetching at d = 256, see the launcher), persistent over tiles,
// op(W) staged once per block in LDS.
//  - Layout.  The MFMA computes the transpose (W fragments as its A operand,
//    the rows as its B operand), so lane (c, g) ends with 4 consecutive
//    columns 16 nb + 4 g of row c and the epilogue moves 16 bytes per lane.
//    Lane (c, g) holds columns 16 kb + 4 g .. + 3 of its row (kb = 0..D/16-1,
//    one float4 each); the K block kb2 of 32 takes the lane's columns from
//    kb = 2 kb2 (slots 0-3) and 2 kb2 + 1 (slots 4-7), and LDS holds op(W)
//    with the same K permutation: uint4 element (kb2 NB + nb) 64 + lane is
//    op(W)[k][16 nb + c] for the lane's 8 K slots, fp16 high parts, then the
//    same array of remainders.
//  - Scaling.  Each row is scaled by the power of two of its largest |x| (the
//    4 lanes of a row agree by two xor shuffles), op(W) by that of its
//    largest |w| (a block reduction while it is staged).
//  - Pipelining.  The next tile's A rows are loaded while the current tile is
//    multiplied, into the other of two register sets (the tile loop is
//    unrolled by two, so no prefetched value is copied: a copy would wait for
//    the load); row-list entries of A are read two tiles ahead, the output
//    rows' one tile ahead; output columns go in groups of NG blocks whose
//    epilogue operands are loaded before their MFMAs and stored right after.
// The loader's fetch_row issues the loads; operand4 turns them into MFMA
// operands (mask, conversion) when they are used.
// kT threads per block, kPF: the next tile's A rows loaded while the current
// one is multiplied (else each wave loads its rows and waits for them, and
// the other waves of the compute unit cover the wait: at d = 256 one block
// of 1024 threads, four waves per SIMD, within 128 VGPRs).
template <int D, bool kTransW, class ALoad, class Epi, bool kListA, bool kListO, int NG, int kMinWaves = (D > 128 ? 2 : 4),
          int kT = kGemmThreads, bool kPF = true>
__global__ void __launch_bounds__(kT, kMinWaves) k_gemm_rows_pp(int64_t n_rows, const float* __restrict__ W,
                                                                ALoad aload, Epi epi) {
  static_assert(D == 64 || D == 128 || D == 256, "pipelined gemm_rows: d = 64, 128 or 256");
  constexpr int DN = F32Slice<D>::DN;
  constexpr int KB = D / 16, KB2 = D / 32, NB = DN / 16;
  static_assert(!Epi::kMask || D == DN, "mask words need the whole row in one block");
  static_assert(NB % NG == 0, "column groups must divide the column blocks");
  static_assert(!Epi::kAddA || !kListO, "an addend taken from A needs the output rows to be the A rows");
  // rows stored in bfloat16 are exact fp16 high parts after the power-of-two
  // scaling (8 significant bits; elements below 2^-32 of the row's largest
  // lose bits of order 2^-38 of it), so their remainder products are skipped
  constexpr bool kHiOnly = HalfRows<ALoad>::value;
  constexpr int kRowsPerTile = 16 * (kT / 64);
  constexpr int kFrag = KB2 * NB * 64;
  extern __shared__ uint4 wfr[];  // [kFrag] high parts, then [kFrag] low parts
  constexpr int kWaves = kT / 64;
  __shared__ float wmax[kWaves + 1];  // per-wave maxima, then the unscale factor of op(W)
  const int tid = threadIdx.x;
  // Block -> (column slice, tile group).  With two slices the blocks that
  // share a tile group differ by 8 in block index, so they run on the same
  // XCD (blocks go round-robin over the 8) at about the same time and the
  // second read of each A row hits its L2.
  const int slice = (D == DN) ? 0 : (int)((blockIdx.x >> 3) & 1);
  const int64_t bgroup = (D == DN) ? (int64_t)blockIdx.x : (int64_t)(((blockIdx.x >> 4) << 3) | (blockIdx.x & 7));
  const int col0 = DN * slice;
  // largest |w| of op(W) (= of W)
  {
    float m = 0.f;
    for (int e = tid; e < D * D / 4; e += kT) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(W + 4 * e);
      m = fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if ((tid & 63) == 0) wmax[tid >> 6] = m;
    __syncthreads();
    m = wmax[0];
#pragma unroll
    for (int q = 1; q < kWaves; ++q) m = fmaxf(m, wmax[q]);
    const uint32_t ew = split_exp(m);
    const float sw = split_scale(ew);
    for (int e = tid; e < kFrag; e += kT) {
      const int l = e & 63;
      const int nb = (e >> 6) % NB;
      const int kb2 = (e >> 6) / NB;
      const int j = col0 + 16 * nb + (l & 15);
      float v[8];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k0 = 16 * (2 * kb2 + h) + 4 * (l >> 4);
        if (kTransW) {
          const f32x4 x = *reinterpret_cast<const f32x4*>(W + (int64_t)j * D + k0);
#pragma unroll
          for (int q = 0; q < 4; ++q) v[4 * h + q] = x[q] * sw;
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) v[4 * h + q] = W[(int64_t)(k0 + q) * D + j] * sw;
        }
      }
      split8(v, wfr[e], wfr[kFrag + e]);
    }
    if (tid == 0) wmax[kWaves] = split_unscale(ew);
    __syncthreads();
  }
  const float uw = wmax[kWaves];
  const int w = tid >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  const int64_t ntiles = (n_rows + kRowsPerTile - 1) / kRowsPerTile;
  const int64_t G = (D == DN) ? (int64_t)gridDim.x : (int64_t)(gridDim.x >> 1);
  typedef RowMap::Key<kListA> KA;
  typedef RowMap::Key<kListO> KO;
  typedef typename ALoad::RowRaw RR;
  // lane (c, g) of wave w owns row 16 w + c of a tile; rows past the end are
  // read from the last row and never stored
  auto row_in = [&](int64_t t) -> int64_t {
    const int64_t i = t * kRowsPerTile + 16 * w + c;
    return i < n_rows ? i : n_rows - 1;
  };
  auto tile = [&](int64_t t, const RR& x, KA ka, KO ko) {
    const int64_t i = t * kRowsPerTile + 16 * w + c;
    const bool live = i < n_rows;
    const int64_t ro = epi.map.template row_of<kListO>(ko);
    const int64_t ra = aload.map.template row_of<kListA>(ka);
    bool rflag = false;
    if constexpr (EpiRowFlag<Epi>::value) rflag = live && epi.flag(ro);
    // the row as MFMA operand: scaled by a power of two of its largest
    // magnitude (or of a bound of it: the stored row, for loaders whose
    // operand only zeroes elements of it), split in two
    uint4 xh[KB2], xlo[KB2];
    // with two column slices, the addend's half of the row (picked once, so
    // the other half's registers are free during the products)
    constexpr bool kHalfAdd = Epi::kAddA && D == 2 * DN;
    typename ALoad::Raw xadd[kHalfAdd ? NB : 1];
    float ux;
    {
      auto absmax4 = [](f32x4 v) { return fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))); };
      float m = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        m = fmaxf(m, absmax4(ALoad::kBoundByStored ? aload.stored4(x, kb) : aload.operand4(x, kb, g)));
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      const uint32_t ex = split_exp(m);
      const float sx = split_scale(ex);
      ux = split_unscale(ex);
#pragma unroll
      for (int kb2 = 0; kb2 < KB2; ++kb2) {
        const f32x4 a0 = aload.operand4(x, 2 * kb2, g), a1 = aload.operand4(x, 2 * kb2 + 1, g);
        // with two column slices, the two blocks of a tile group load the
        // same A rows: each writes the half of the row in its own columns
        if (ALoad::kTee && live && (D == DN || (2 * kb2 < KB2) == (slice == 0))) {
          aload.tee4(ra, 2 * kb2, g, a0);
          aload.tee4(ra, 2 * kb2 + 1, g, a1);
        }
        float v[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[q] = a0[q] * sx;
          v[4 + q] = a1[q] * sx;
        }
        if constexpr (kHalfAdd) {
          // K blocks 2 kb2 and 2 kb2 + 1 hold output columns of slice 0 when
          // kb2 < KB2 / 2, of slice 1 otherwise
          if (2 * kb2 < NB) {
            xadd[2 * kb2] = slice == 0 ? x.x[2 * kb2] : x.x[NB + 2 * kb2];
            xadd[2 * kb2 + 1] = slice == 0 ? x.x[2 * kb2 + 1] : x.x[NB + 2 * kb2 + 1];
          }
        }
        if constexpr (kHiOnly) {
          uint32_t h[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) h[q] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(v[2 * q], v[2 * q + 1]));
          xh[kb2] = uint4{h[0], h[1], h[2], h[3]};
        } else {
          split8(v, xh[kb2], xlo[kb2]);
        }
      }
    }
#pragma unroll
    for (int p = 0; p < NB / NG; ++p) {
      // without prefetching (128 VGPRs) each column group's W fragments are
      // read where they are used, not hoisted ahead of earlier groups
      if constexpr (!kPF) __builtin_amdgcn_sched_barrier(0);
      f32x4 pre[NG];
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        const int col = col0 + 16 * (p * NG + q) + 4 * g;
        if constexpr (Epi::kAddA) {
          // output column block col0/16 + p NG + q covers the lane's A columns of that K block
          // (both candidate blocks are named at compile time: a run-time index
          // would send the row's registers to memory)
          f32x4 st;
          if constexpr (D == DN) {
            st = aload.stored4(x, p * NG + q);
          } else {
            static_assert(D == 2 * DN, "two column slices");
            st = aload.stored4r(xadd[p * NG + q]);
          }
          pre[q] = epi.addend ? epi.bias4(col) + st : epi.bias4(col);
        } else {
          pre[q] = epi.pre4(i, ro, col);
        }
      }
      f32x4 acc[NG];
#pragma unroll
      for (int q = 0; q < NG; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb2 = 0; kb2 < KB2; ++kb2) {
#pragma unroll
        for (int q = 0; q < NG; ++q) {
          const int e = (kb2 * NB + p * NG + q) * 64 + l;
          const uint4 bh = wfr[e], bl = wfr[kFrag + e];
          acc[q] = mfma_f16(bh, xh[kb2], acc[q]);
          if constexpr (!kHiOnly) acc[q] = mfma_f16(bh, xlo[kb2], acc[q]);
          acc[q] = mfma_f16(bl, xh[kb2], acc[q]);
        }
        // the residual's half row stays live through the products: W
        // fragments are read at most four K blocks ahead
        if constexpr (!kPF && kHalfAdd) {
          if (kb2 % 4 == 3) __builtin_amdgcn_sched_barrier(0);
        }

      }
#pragma unroll
      for (int q = 0; q < NG; ++q) acc[q] = split_unscale4(acc[q], ux, uw);
      if constexpr (Epi::kMask) {
        // store4 returns the 4 output-decision bits of its columns; the lanes
        // (c, 0..3) of a 32-column group hold one 32-bit mask word together
        static_assert(NG == 2, "mask words need 32-column groups");
        uint32_t word = 0;
#pragma unroll
        for (int q = 0; q < NG; ++q) {
          const uint32_t nib = live ? epi.store4(i, ro, col0 + 16 * (p * NG + q) + 4 * g, acc[q], pre[q]) : 0u;
          word |= nib << (16 * q + 4 * g);
        }
        word |= __shfl_xor(word, 16, 64);
        word |= __shfl_xor(word, 32, 64);
        if (live && g == 0) epi.mask_word(ro, p, word);
      } else if (live) {
#pragma unroll
        for (int q = 0; q < NG; ++q) {
          if constexpr (EpiRowFlag<Epi>::value) {
            epi.store4f(i, ro, col0 + 16 * (p * NG + q) + 4 * g, acc[q], pre[q], rflag);
          } else {
            epi.store4(i, ro, col0 + 16 * (p * NG + q) + 4 * g, acc[q], pre[q]);
          }
        }
      }
    }
  };
  int64_t t = bgroup;
  if (t >= ntiles) return;
  if constexpr (!kPF) {
    for (; t < ntiles; t += G) {
      const KA ka = aload.map.template key<kListA>(row_in(t));
      const KO ko = epi.map.template key<kListO>(row_in(t));
      RR x;
      aload.fetch_row(aload.map.template row_of<kListA>(ka), g, x);
      tile(t, x, ka, ko);
    }
    return;
  }
  KA ka0 = aload.map.template key<kListA>(row_in(t));
  KA ka1 = aload.map.template key<kListA>(row_in(t + G));
  KO ko0 = epi.map.template key<kListO>(row_in(t));
  KO ko1;
  RR x0, x1;
  aload.fetch_row(aload.map.template row_of<kListA>(ka0), g, x0);
  // the body handles tiles t and t + G (the second may lie past the end: its
  // rows are clamped and nothing is stored)
  for (; t < ntiles; t += 2 * G) {
    {
      const KA kc = ka0;
      aload.fetch_row(aload.map.template row_of<kListA>(ka1), g, x1);
      ka0 = aload.map.template key<kListA>(row_in(t + 2 * G));
      ko1 = epi.map.template key<kListO>(row_in(t + G));
      __builtin_amdgcn_sched_barrier(0);
      tile(t, x0, kc, ko0);
      __builtin_amdgcn_sched_barrier(0);
    }
    {
      const KA kc = ka1;
      aload.fetch_row(aload.map.template row_of<kListA>(ka0), g, x0);
      ka1 = aload.map.template key<kListA>(row_in(t + 3 * G));
      ko0 = epi.map.template key<kListO>(row_in(t + 2 * G));
      __builtin_amdgcn_sched_barrier(0);
      tile(t + G, x1, kc, ko1);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

constexpr int kGemmPPBlocksPerCu = 2;
template <int D, bool kTransW, class ALoad, class Epi>
int launch_gemm_rows_pp(const char* name, int64_t n_rows, const float* W, ALoad aload, Epi epi, hipStream_t s) {
  if (n_rows <= 0) return HG_OK;
  // the masked loader's rows (with their mask words) are the largest prefetch
  // and, as the residual addend, may stay live through the tile: one column
  // block per group keeps it within 128 VGPRs
  // d = 256: one block of 1024 threads per compute unit (its LDS slice of
  // op(W) takes 128 KB), no prefetch, 128 VGPRs -- except float32 rows held
  // as the residual addend (64 VGPRs on top of their split parts), which keep
  // the 512-thread prefetching kernel
  constexpr bool kBig = D == 256 && !(Epi::kAddA && sizeof(typename ALoad::Raw) == 16);
  constexpr int NG = (ALoad::kTee && (D == 128 || (Epi::kAddA && sizeof(typename ALoad::Raw) == 16))) ? 1 : 2;
  // float32 masked rows at d = 128 holding the residual addend: 256 VGPRs,
  // one block per compute unit (the residual is not read a second time)
  constexpr bool kWide = ALoad::kTee && Epi::kAddA && D == 128 && sizeof(typename ALoad::Raw) == 16;
  constexpr int kT = kBig ? 2 * kGemmThreads : kGemmThreads;
  constexpr int kMinWaves = kBig ? 1 : ((D > 128 || kWide) ? 2 : 4);
  constexpr int DN = F32Slice<D>::DN;
  const int64_t tiles = cdiv(n_rows, 16 * (kT / 64));
  // LDS holds a D x DN slice of op(W): 64 KB up to d = 128 (two resident
  // blocks per compute unit), 128 KB at d = 256 (one)
  const int64_t cap = (int64_t)num_cus() * ((D > 128 || kWide) ? 1 : kGemmPPBlocksPerCu);
  int64_t grid = tiles < cap ? tiles : cap;
  // two column slices: 2 blocks per tile group, groups in multiples of 8 (the
  // kernel's block -> (slice, group) map pairs blocks 16 q + x and 16 q + 8 + x)
  if (D > DN) grid = 2 * (cdiv(tiles < cap / 2 ? tiles : cap / 2, 8) * 8);
  const size_t lds = sizeof(float) * D * DN;
  const bool la = aload.map.list != nullptr, lo = epi.map.list != nullptr;
#define HG_PP_LAUNCH(LA_, LO_)                                                                          \
  do {                                                                                                  \
    auto kern = k_gemm_rows_pp<D, kTransW, ALoad, Epi, LA_, LO_, NG, kMinWaves, kT, !kBig>;             \
    if (lds > 65536) {                                                                                  \
      static bool attr_set = false;                                                                     \
      if (!attr_set) {                                                                                  \
        HG_HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void*>(kern),                             \
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));          \
        attr_set = true;                                                                                \
      }                                                                                                 \
    }                                                                                                   \
    HG_LAUNCH(name, kern, dim3((unsigned)grid), dim3(kT), lds, s, n_rows, W, aload, epi);                   \
  } while (0)
  if constexpr (Epi::kAddA) {
    // the addend is read from the A registers: output row i must be A row i
    if (la || lo || aload.map.first != epi.map.first || aload.map.mul != epi.map.mul ||
        aload.map.add != epi.map.add)
      return fail(HG_ERR_ARG, "%s: an addend taken from A needs identical contiguous row maps", name);
    HG_PP_LAUNCH(false, false);
  } else {
    if (la && lo) {
      HG_PP_LAUNCH(true, true);
    } else if (la) {
      HG_PP_LAUNCH(true, false);
    } else if (lo) {
      HG_PP_LAUNCH(false, true);
    } else {
      HG_PP_LAUNCH(false, false);
    }
  }
#undef HG_PP_LAUNCH
  return HG_OK;
}

// ---- gemm_rows, bfloat16 MFMA ----------------------------------------------------
// v_mfma_f32_16x16x32_bf16: lane (c, g) supplies A[row c][32 kb + 8 g + e],
// e = 0..7 -- eight consecutive columns, one 16-byte load -- and
// op(W)[32 kb + 8 g + e][16 nb + c] from LDS, where op(W) is staged rounded to
// bfloat16 in fragment order (uint4 element (kb*NB + nb)*64 + lane).  A block
// is RG row groups x CG column groups of waves; a wave owns 16 rows and D/CG
// columns.  Accumulation is float32.
template <int D>
struct BfShape {
  // one wave per 16 rows and all D columns: each A row is read by one wave
  // only (column groups of waves sharing rows fetched them from memory up to
  // 2.4 times at d = 256)
  static constexpr int CG = 1;
  static constexpr int RG = 8;
  static constexpr int kThreads = 64 * CG * RG;
};

template <int D, bool kTransW, class ALoad, class Epi>
__global__ void __launch_bounds__(BfShape<D>::kThreads) k_gemm_rows_bf16(int64_t n_rows, const float* __restrict__ W,
                                                                       ALoad aload, Epi epi) {
  constexpr int NB = D / 16, KB = D / 32;
  constexpr int CG = BfShape<D>::CG, RG = BfShape<D>::RG, NT = BfShape<D>::kThreads;
  constexpr int NBW = NB / CG;
  extern __shared__ uint4 wlb[];
  const int tid = threadIdx.x;
  for (int e = tid; e < KB * NB * 64; e += NT) {
    const int l = e & 63;
    const int nb = (e >> 6) % NB;
    const int kb = (e >> 6) / NB;
    const int j = 16 * nb + (l & 15);
    const int k0 = 32 * kb + 8 * (l >> 4);
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = kTransW ? W[(int64_t)j * D + k0 + q] : W[(int64_t)(k0 + q) * D + j];
    wlb[e] = uint4{pack2bf(v[0], v[1]), pack2bf(v[2], v[3]), pack2bf(v[4], v[5]), pack2bf(v[6], v[7])};
  }
  __syncthreads();
  const int w = tid >> 6;
  const int rg = w / CG, cg = w % CG;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  constexpr int kRowsPerTile = 16 * RG;
  const int64_t ntiles = (n_rows + kRowsPerTile - 1) / kRowsPerTile;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t r0 = t * kRowsPerTile + 16 * rg;
    uint4 a[KB];
    {
      const int64_t ia = r0 + c;
      if (ia < n_rows) {
        const auto p = aload.rowp(ia);
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) a[kb] = aload.load8bf(p, 32 * kb + 8 * g);
      } else {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) a[kb] = uint4{0u, 0u, 0u, 0u};
      }
    }
    f32x4 acc[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nb0 = 0; nb0 < NBW; nb0 += 4) {
        uint4 b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) b[u] = wlb[(kb * NB + cg * NBW + nb0 + u) * 64 + l];
        // transposed product: W fragments as the A operand, A rows as the B operand
#pragma unroll
        for (int u = 0; u < 4; ++u) acc[nb0 + u] = mfma_bf16(b[u], a[kb], acc[nb0 + u]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    // lane (c, g) holds row r0 + c, columns 16 (cg*NBW + nb) + 4 g .. + 3
    const int64_t i = r0 + c;
    if (i < n_rows) {
      const int64_t ro = epi.row(i);
      f32x4 pre[NBW];
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) pre[nb] = epi.pre4(i, ro, 16 * (cg * NBW + nb) + 4 * g);
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) epi.store4(i, ro, 16 * (cg * NBW + nb) + 4 * g, acc[nb], pre[nb]);
    }
  }
}

template <int D, bool kTransW, class ALoad, class Epi>
int launch_gemm_rows_bf16(const char* name, int64_t n_rows, const float* W, ALoad aload, Epi epi,
                          hipStream_t s) {
  if (n_rows <= 0) return HG_OK;
  const int64_t tiles = cdiv(n_rows, 16 * BfShape<D>::RG);
  const int64_t cap = (int64_t)num_cus() * (D >= 256 ? 1 : 2);
  const int64_t grid = tiles < cap ? tiles : cap;
  const size_t lds = sizeof(uint16_t) * D * D;
  auto kern = k_gemm_rows_bf16<D, kTransW, ALoad, Epi>;
  if (lds > 65536) {
    static bool attr_set = false;
    if (!attr_set) {
      HG_HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
      attr_set = true;
    }
  }
  HG_LAUNCH(name, kern, dim3((unsigned)grid), dim3(BfShape<D>::kThreads), lds, s, n_rows, W, aload, epi);
  return HG_OK;
}

// ---- gemm_tn split-K ----------------------------------------------------------
// Split-K block -> (chunk, output tile).  At d = 256 the output is four
// 128 x 128 tiles (ti, tj) that read the same rows of a chunk: the four blocks
// of a chunk are 8 apart in groups of 32 consecutive blocks, so they go to the
// same XCD (blocks are dealt round-robin over the 8) at about the same time
// and the rows come from HBM once, then from that XCD's L2.  The grid covers
// the chunk count rounded up to 8; a block past the last chunk has no rows.
template <int D>
__device__ __forceinline__ void tn_block(int64_t& chunk, int& ti, int& tj) {
  if constexpr (D == 256) {
    const unsigned b = blockIdx.x;
    const int t = (int)((b >> 3) & 3u);
    chunk = (int64_t)(((b >> 5) << 3) | (b & 7u));
    ti = t >> 1;
    tj = t & 1;
  } else {
    chunk = blockIdx.x;
    ti = tj = 0;
  }
}
inline unsigned tn_grid(int D, int64_t chunks) {
  return (unsigned)(D == 256 ? 4 * cdiv(chunks, 8) * 8 : chunks);
}

// partial[chunk][i][j] = sum_{rows k of the chunk} A[k][i] * B[k][j]
// colsum[chunk][j]    = sum_{rows k of the chunk} B[k][j]        (if colsum)
// A wave owns a 64 x 64 block of the output (D = 128: wave w takes quadrant
// (w/2, w%2) over every row of the chunk; D = 64: every wave takes the whole
// output over every fourth group of 4 rows, and the waves are summed in LDS
// in wave order).  Lane (c, g) reads one float4 of A and of B per row
// (features q0 + 4c .. 4c+3) and feeds component b of it to MFMA block b, so
// block b, MFMA index c stands for feature q0 + 4c + b: in the output, the
// lane's register v of block (bi, bj) is element [4 (4 g + v) + bi][4 c + bj].
template <int D, class LA, class LB, bool kListA, bool kListB>
__global__ void __launch_bounds__(256) k_gemm_tn(int64_t n_rows, int64_t kc, LA la, LB lb,
                                                 float* __restrict__ partial,
                                                 float* __restrict__ colsum) {
  static_assert(D == 64 || D == 128 || D == 256, "gemm_tn: d must be 64, 128 or 256");
  constexpr bool kQuad = (D >= 128);
  const int w = threadIdx.x >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  int64_t chunk;
  int ti, tj;
  tn_block<D>(chunk, ti, tj);
  const int64_t k_beg = chunk * kc;
  if (k_beg >= n_rows) return;  // a padding block (the whole block)
  const int64_t k_end = (k_beg + kc < n_rows) ? k_beg + kc : n_rows;
  const int qi = kQuad ? (w >> 1) : 0;
  const int qj = kQuad ? (w & 1) : 0;
  const int64_t step0 = kQuad ? 0 : 4 * w;
  const int64_t stride = kQuad ? 4 : 16;
  const int ca = 128 * ti + 64 * qi + 4 * c, cb = 128 * tj + 64 * qj + 4 * c;
  f32x4 acc[4][4];
  f32x4 bs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 4; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Software pipeline over steps of U row groups: the rows of step s + 1 are
  // loaded and the row-list entries of step s + 2 looked up while step s is
  // multiplied.  Two register sets alternate (the loop body is unrolled by
  // two), so no prefetched value is ever copied.  Rows past the chunk end are
  // read from its last row and zeroed before use.
  constexpr int U = 4;
  typedef typename LA::Raw RA;
  typedef typename LB::Raw RB;
  const int64_t S = stride * U;
  const typename LA::Prep pa = la.prep(ca);
  const typename LB::Prep pb = lb.prep(cb);
  typedef RowMap::Key<kListA> KA;
  typedef RowMap::Key<kListB> KB;
  auto keys = [&](int64_t k0, KA (&ka)[U], KB (&kb)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      int64_t r = k0 + u * stride + g;
      r = r < k_end ? r : k_end - 1;
      ka[u] = la.map.template key<kListA>(r);
      kb[u] = lb.map.template key<kListB>(r);
    }
  };
  auto fetch = [&](const KA (&ka)[U], const KB (&kb)[U], RA (&xa)[U], RB (&xb)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      xa[u] = la.raw4b(la.map.template row_of<kListA>(ka[u]), ca);
      xb[u] = lb.raw4b(lb.map.template row_of<kListB>(kb[u]), cb);
    }
  };
  auto compute = [&](int64_t k0, const RA (&xa)[U], const RB (&xb)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool ok = k0 + u * stride + g < k_end;
      f32x4 a = la.cook4(xa[u], pa), b = lb.cook4(xb[u], pb);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = ok ? a[q] : 0.f;
        b[q] = ok ? b[q] : 0.f;
      }
      bs += b;
#pragma unroll
      for (int bi = 0; bi < 4; ++bi)
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) acc[bi][bj] = mfma4(a[bi], b[bj], acc[bi][bj]);
    }
  };
  int64_t k0 = k_beg + step0;
  if (k0 < k_end) {
    KA k0a[U], k1a[U];
    KB k0b[U], k1b[U];
    RA x0a[U], x1a[U];
    RB x0b[U], x1b[U];
    keys(k0, k0a, k0b);
    fetch(k0a, k0b, x0a, x0b);
    keys(k0 + S, k1a, k1b);
    // one basic block per pair of steps (a second step past the chunk end
    // multiplies zeroed rows); the barriers keep each phase where it is
    for (; k0 < k_end; k0 += 2 * S) {
      fetch(k1a, k1b, x1a, x1b);
      keys(k0 + 2 * S, k0a, k0b);
      __builtin_amdgcn_sched_barrier(0);
      compute(k0, x0a, x0b);
      __builtin_amdgcn_sched_barrier(0);
      fetch(k0a, k0b, x0a, x0b);
      keys(k0 + 3 * S, k1a, k1b);
      __builtin_amdgcn_sched_barrier(0);
      compute(k0 + S, x1a, x1b);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // column sums: reduce the 4 row groups of the wave
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    bs[q] += __shfl_xor(bs[q], 16, 64);
    bs[q] += __shfl_xor(bs[q], 32, 64);
  }
  float* out = partial + chunk * (int64_t)D * D;
  if (kQuad) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t i = 128 * ti + 64 * qi + 4 * (4 * g + v) + bi;
        f32x4 row4;
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) row4[bj] = acc[bi][bj][v];
        *reinterpret_cast<f32x4*>(out + i * D + cb) = row4;
      }
    if (colsum && ti == 0 && qi == 0 && g == 0) *reinterpret_cast<f32x4*>(colsum + chunk * D + cb) = bs;
  } else {
    __shared__ float red[64 * 64];
    __shared__ float cred[64];
    for (int ww = 0; ww < 4; ++ww) {
      if (w == ww) {
#pragma unroll
        for (int bi = 0; bi < 4; ++bi)
#pragma unroll
          for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int bj = 0; bj < 4; ++bj) {
              const int idx = (4 * (4 * g + v) + bi) * 64 + 4 * c + bj;
              red[idx] = (ww == 0 ? 0.f : red[idx]) + acc[bi][bj][v];
            }
        if (g == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) cred[4 * c + q] = (ww == 0 ? 0.f : cred[4 * c + q]) + bs[q];
        }
      }
      __syncthreads();
    }
    for (int e = threadIdx.x; e < 64 * 64; e += 256) out[e] = red[e];
    if (colsum && threadIdx.x < 64) colsum[chunk * D + threadIdx.x] = cred[threadIdx.x];
  }
}

// Two float32 values -> three bf16 parts each (packed pairs, round to nearest
// even): v = p0 + p1 + p2 + r with |r| <= 2^-24 |v| (each part carries the
// next 8 significant bits of what the previous ones left).
__device__ __forceinline__ void split_bf3(float v0, float v1, uint32_t (&part)[3]) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const bf16x2_t h = {(__bf16)v0, (__bf16)v1};
    part[k] = __builtin_bit_cast(uint32_t, h);
    v0 -= __uint_as_float(part[k] << 16);
    v1 -= __uint_as_float(part[k] & 0xFFFF0000u);
  }
}

// gemm_tn on v_mfma_f32_16x16x32_bf16 for plain feature rows, K = 32 rows
// per step: lane (c, g) reads rows 8 g .. 8 g + 7 of the step (one A load and
// one B load of 4 features each per row), and block b of an operand is
// feature ca + 4 c + b (cb + 4 c + b) of those 8 rows, as in k_gemm_tn.
// Rows stored in bfloat16 are exact MFMA operands; float32 rows are split
// into three bf16 parts (split_bf3, 2^-24 of each element left over).  Per
// block pair: one MFMA (bf16 x bf16), three (one side split: the bf16 side
// times each part) or six (both split: every part product of order <= 2,
// p0 q0, p0 q1, p1 q0, p0 q2, p2 q0, p1 q1; the dropped ones are below
// 2^-24 of the product), at a fraction of the float32 MFMA's cost with
// float32-like products.  Same outputs, chunking, wave tiling and epilogue
// as k_gemm_tn.
template <int D, class TA, class TB, bool kListA, bool kListB>
__global__ void __launch_bounds__(256, 2) k_gemm_tn_bf(int64_t n_rows, int64_t kc, LoadRows<D, TA> la,
                                                       LoadRows<D, TB> lb, float* __restrict__ partial,
                                                       float* __restrict__ colsum) {
  static_assert(D == 64 || D == 128 || D == 256, "gemm_tn_bf: d must be 64, 128 or 256");
  constexpr bool kQuad = (D >= 128);
  constexpr bool kSplitA = sizeof(TA) == 4;
  constexpr bool kSplitB = sizeof(TB) == 4;
  constexpr int E = 8;  // rows per lane and step
  const int w = threadIdx.x >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  int64_t chunk;
  int ti, tj;
  tn_block<D>(chunk, ti, tj);
  const int64_t k_beg = chunk * kc;
  if (k_beg >= n_rows) return;  // a padding block (the whole block)
  const int64_t k_end = (k_beg + kc < n_rows) ? k_beg + kc : n_rows;
  const int qi = kQuad ? (w >> 1) : 0;
  const int qj = kQuad ? (w & 1) : 0;
  const int64_t step0 = kQuad ? 0 : 32 * w;
  const int64_t S = kQuad ? 32 : 128;
  const int ca = 128 * ti + 64 * qi + 4 * c, cb = 128 * tj + 64 * qj + 4 * c;
  f32x4 acc[4][4];
  f32x4 bs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 4; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};
  typedef typename Elt<TA>::raw4_t RA;
  typedef typename Elt<TB>::raw4_t RB;
  typedef RowMap::Key<kListA> KA;
  typedef RowMap::Key<kListB> KB;
  auto keys = [&](int64_t k0, KA (&ka)[E], KB (&kb)[E]) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      int64_t r = k0 + 8 * g + e;
      r = r < k_end ? r : k_end - 1;
      ka[e] = la.map.template key<kListA>(r);
      kb[e] = lb.map.template key<kListB>(r);
    }
  };
  auto fetch = [&](const KA (&ka)[E], const KB (&kb)[E], RA (&xa)[E], RB (&xb)[E]) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      xa[e] = la.raw4b(la.map.template row_of<kListA>(ka[e]), ca);
      xb[e] = lb.raw4b(lb.map.template row_of<kListB>(kb[e]), cb);
    }
  };
  // rows 2p, 2p + 1 of bf16 feature f (of 4 per raw uint2) as one bf16 pair
  auto pair_bf = [](uint2 x0, uint2 x1, int f) -> uint32_t {
    const uint32_t a = (f < 2) ? x0.x : x0.y, b = (f < 2) ? x1.x : x1.y;
    return (f & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
  };
  auto compute = [&](int64_t k0, const RA (&xa0)[E], const RB (&xb0)[E]) {
    RA xa[E];
    RB xb[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const bool ok = k0 + 8 * g + e < k_end;
      if constexpr (kSplitA) {
        xa[e] = ok ? xa0[e] : RA{0.f, 0.f, 0.f, 0.f};
      } else {
        xa[e] = ok ? xa0[e] : RA{0u, 0u};
      }
      if constexpr (kSplitB) {
        xb[e] = ok ? xb0[e] : RB{0.f, 0.f, 0.f, 0.f};
      } else {
        xb[e] = ok ? xb0[e] : RB{0u, 0u};
      }
    }
    constexpr int PA = kSplitA ? 3 : 1, PB = kSplitB ? 3 : 1;
    uint4 bq[4][PB];
#pragma unroll
    for (int bj = 0; bj < 4; ++bj) {
      uint32_t w[PB][4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        if constexpr (kSplitB) {
          const float v0 = xb[2 * p][bj], v1 = xb[2 * p + 1][bj];
          bs[bj] += v0 + v1;
          uint32_t part[3];
          split_bf3(v0, v1, part);
#pragma unroll
          for (int k = 0; k < 3; ++k) w[k][p] = part[k];
        } else {
          w[0][p] = pair_bf(xb[2 * p], xb[2 * p + 1], bj);
          bs[bj] += __uint_as_float(w[0][p] << 16) + __uint_as_float(w[0][p] & 0xFFFF0000u);
        }
      }
#pragma unroll
      for (int k = 0; k < PB; ++k) bq[bj][k] = uint4{w[k][0], w[k][1], w[k][2], w[k][3]};
    }
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) {
      uint4 aq[PA];
      if constexpr (kSplitA) {
        uint32_t w[3][4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          uint32_t part[3];
          split_bf3(xa[2 * p][bi], xa[2 * p + 1][bi], part);
#pragma unroll
          for (int k = 0; k < 3; ++k) w[k][p] = part[k];
        }
#pragma unroll
        for (int k = 0; k < 3; ++k) aq[k] = uint4{w[k][0], w[k][1], w[k][2], w[k][3]};
      } else {
        aq[0] = uint4{pair_bf(xa[0], xa[1], bi), pair_bf(xa[2], xa[3], bi), pair_bf(xa[4], xa[5], bi),
                      pair_bf(xa[6], xa[7], bi)};
      }
#pragma unroll
      for (int bj = 0; bj < 4; ++bj) {
        // part products of order pa + pb <= 2, smallest first
#pragma unroll
        for (int ord = 2; ord >= 0; --ord)
#pragma unroll
          for (int pa = 0; pa < PA; ++pa) {
            const int pb = ord - pa;
            if (pb >= 0 && pb < PB) acc[bi][bj] = mfma_bf16(aq[pa], bq[bj][pb], acc[bi][bj]);
          }
      }
    }
  };
  int64_t k0 = k_beg + step0;
  if (k0 < k_end) {
    KA k0a[E], k1a[E];
    KB k0b[E], k1b[E];
    keys(k0, k0a, k0b);
    if constexpr (kSplitA && kSplitB) {
      // float32 rows on both sides: their split parts take the registers of
      // a second row set, so rows are not prefetched (the other waves of the
      // compute unit cover the load latency); row-list entries still are
      RA xa[E];
      RB xb[E];
      for (; k0 < k_end; k0 += S) {
        fetch(k0a, k0b, xa, xb);
        keys(k0 + S, k1a, k1b);
        __builtin_amdgcn_sched_barrier(0);
        compute(k0, xa, xb);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          k0a[e] = k1a[e];
          k0b[e] = k1b[e];
        }
      }
    } else {
      RA x0a[E], x1a[E];
      RB x0b[E], x1b[E];
      fetch(k0a, k0b, x0a, x0b);
      keys(k0 + S, k1a, k1b);
      // one basic block per pair of steps (a second step past the chunk end
      // multiplies zeroed rows); the barriers keep each phase where it is
      for (; k0 < k_end; k0 += 2 * S) {
        fetch(k1a, k1b, x1a, x1b);
        keys(k0 + 2 * S, k0a, k0b);
        __builtin_amdgcn_sched_barrier(0);
        compute(k0, x0a, x0b);
        __builtin_amdgcn_sched_barrier(0);
        fetch(k0a, k0b, x0a, x0b);
        keys(k0 + 3 * S, k1a, k1b);
        __builtin_amdgcn_sched_barrier(0);
        compute(k0 + S, x1a, x1b);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // column sums: reduce the 4 row groups of the wave
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    bs[q] += __shfl_xor(bs[q], 16, 64);
    bs[q] += __shfl_xor(bs[q], 32, 64);
  }
  float* out = partial + chunk * (int64_t)D * D;
  if (kQuad) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t i = 128 * ti + 64 * qi + 4 * (4 * g + v) + bi;
        f32x4 row4;
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) row4[bj] = acc[bi][bj][v];
        *reinterpret_cast<f32x4*>(out + i * D + cb) = row4;
      }
    if (colsum && ti == 0 && qi == 0 && g == 0) *reinterpret_cast<f32x4*>(colsum + chunk * D + cb) = bs;
  } else {
    __shared__ float red[64 * 64];
    __shared__ float cred[64];
    for (int ww = 0; ww < 4; ++ww) {
      if (w == ww) {
#pragma unroll
        for (int bi = 0; bi < 4; ++bi)
#pragma unroll
          for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int bj = 0; bj < 4; ++bj) {
              const int idx = (4 * (4 * g + v) + bi) * 64 + 4 * c + bj;
              red[idx] = (ww == 0 ? 0.f : red[idx]) + acc[bi][bj][v];
            }
        if (g == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) cred[4 * c + q] = (ww == 0 ? 0.f : cred[4 * c + q]) + bs[q];
        }
      }
      __syncthreads();
    }
    for (int e = threadIdx.x; e < 64 * 64; e += 256) out[e] = red[e];
    if (colsum && threadIdx.x < 64) colsum[chunk * D + threadIdx.x] = cred[threadIdx.x];
  }
}

template <class L>
struct IsPlainRows : std::false_type {};
template <int D, class T>
struct IsPlainRows<LoadRows<D, T>> : std::true_type {};

// Fixed-order reduction of nchunks partial arrays of n floats, in two stages:
// group g sums chunks [g*per, (g+1)*per) in order into tmp[g], then the groups
// are summed in order: out[i] (+)= sum_g tmp[g][i].
constexpr int kSplitGroups = 16;

static __global__ void k_sum_partials_grouped(const float* __restrict__ partial, int64_t nchunks,
                                              int64_t n, int64_t per, float* __restrict__ tmp) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t grp = blockIdx.y;
  if (i >= n) return;
  const int64_t c0 = grp * per;
  const int64_t c1 = (c0 + per < nchunks) ? c0 + per : nchunks;
  float s = 0.f;
  for (int64_t c = c0; c < c1; ++c) s += partial[c * n + i];
  tmp[grp * n + i] = s;
}

// out[i] (+)= sum_{c < nchunks} partial[c][i]   (fixed order)
static __global__ void k_sum_partials(const float* __restrict__ partial, int64_t nchunks, int64_t n,
                                      float* __restrict__ out, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = accumulate ? out[i] : 0.f;
  for (int64_t c = 0; c < nchunks; ++c) s += partial[c * n + i];
  out[i] = s;
}

// gemm_tn on v_mfma_f32_16x16x32_bf16 for plain feature rows at d = 128 and
// 256 whose two operands have the same storage type (float32 x float32: each
// element split once per block instead of by each wave that uses it, 2.64 ->
// 2.2 ms per weight gradient of the 10M-row self transform; bf16 x bf16).
// A bf16 x float32 product stays with k_gemm_tn_bf, which measured twice as
// fast at d = 256 (its four independent waves per block keep more rows in
// flight than a block synchronised per step).  The operands are staged in LDS
// once per step.  A block computes one
// 128 x 128 output tile (ti, tj) of its chunk (d = 256: four blocks per
// chunk, as in k_gemm_tn_bf) in steps of 32 rows.  Threads 0-127 stage A,
// 128-255 B: thread u takes rows 8 (u/32) .. + 7 of the step and features
// 4 (u%32) .. + 3 of the tile, one raw load of 4 features per row, and
// writes per feature the 8 rows' values as one uint4 of bf16 -- the MFMA's
// 8 K slots of K group u/32 -- into LDS (float32 rows: the three bf16 parts
// of split_bf3, each element split once per block instead of once per wave
// that uses it).  The next step's rows are loaded while the waves multiply.
// Wave w owns the 64 x 64 quadrant (w/2, w%2) of the tile; MFMA block
// (bi, bj) covers tile rows 64 qi + 16 bi + m and columns 64 qj + 16 bj + n,
// lane (c, g) supplying K group g of A row m = c and B column n = c, and
// holding output (m = 4 g + v, n = c).  Part products of order <= 2,
// smallest first, as in k_gemm_tn_bf.  Same outputs and chunking as
// k_gemm_tn_bf (column sums of B in float32, rows in order per K group, the
// four K groups summed in order).
// A block barrier ordering LDS accesses only: global loads in flight (the
// next step's rows) stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int D, class TA, class TB, bool kListA, bool kListB>
__global__ void __launch_bounds__(256, 2) k_gemm_tn_lds(int64_t n_rows, int64_t kc, LoadRows<D, TA> la,
                                                        LoadRows<D, TB> lb, float* __restrict__ partial,
                                                        float* __restrict__ colsum) {
  static_assert(D == 128 || D == 256, "gemm_tn_lds: d must be 128 or 256");
  constexpr bool kSplitA = sizeof(TA) == 4, kSplitB = sizeof(TB) == 4;
  constexpr int PA = kSplitA ? 3 : 1, PB = kSplitB ? 3 : 1;
  constexpr int TT = 128;  // output tile edge
  constexpr int S = 32;    // rows per step
  __shared__ uint4 fa[PA][4][TT];
  __shared__ uint4 fb[PB][4][TT];
  // feature f's fragment sits at f ^ ((f / 16) mod 4): a staging thread
  // writes 4 consecutive features and its neighbours the next 4, so without
  // the swizzle a store of 32 lanes hits each bank 8 times; with it the
  // stores spread over all banks, and the 16 lanes of a fragment read still
  // find a permutation of 16 consecutive slots
  auto swz = [](int f) { return f ^ ((f >> 4) & 3); };
  __shared__ float cred[4][TT];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int g = l >> 4, c = l & 15;
  int64_t chunk;
  int ti, tj;
  tn_block<D>(chunk, ti, tj);
  const int64_t k_beg = chunk * kc;
  if (k_beg >= n_rows) return;  // a padding block (the whole block)
  const int64_t k_end = (k_beg + kc < n_rows) ? k_beg + kc : n_rows;
  // staging role (uniform per wave)
  const bool sb = tid >= 128;
  const int u = tid & 127, sg = u >> 5, sf = 4 * (u & 31);
  const int scol = (sb ? TT * tj : TT * ti) + sf;
  // row keys of a step: list entries (loaded ahead) or the row index itself
  // (both below 2^31)
  int32_t kk[8];
  auto keys = [&](int64_t k0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      int64_t r = k0 + 8 * sg + e;
      r = r < k_end ? r : k_end - 1;
      if (sb) {
        kk[e] = (int32_t)lb.map.template key<kListB>(r);
      } else {
        kk[e] = (int32_t)la.map.template key<kListA>(r);
      }
    }
  };
  uint4 rawa[8];  // 4 features of each of the 8 rows, as loaded (bf16 rows use .x and .y)
  auto fetch = [&](int64_t k0, uint4 (&raw)[8]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      raw[e] = uint4{0u, 0u, 0u, 0u};
      if (k0 + 8 * sg + e < k_end) {
        if (sb) {
          const int64_t row = lb.map.template row_of<kListB>((typename RowMap::template Key<kListB>)kk[e]);
          if constexpr (kSplitB) {
            raw[e] = __builtin_bit_cast(uint4, lb.raw4b(row, scol));
          } else {
            const uint2 x = lb.raw4b(row, scol);
            raw[e] = uint4{x.x, x.y, 0u, 0u};
          }
        } else {
          const int64_t row = la.map.template row_of<kListA>((typename RowMap::template Key<kListA>)kk[e]);
          if constexpr (kSplitA) {
            raw[e] = __builtin_bit_cast(uint4, la.raw4b(row, scol));
          } else {
            const uint2 x = la.raw4b(row, scol);
            raw[e] = uint4{x.x, x.y, 0u, 0u};
          }
        }
      }
    }
  };
  // feature q of rows 2p, 2p + 1 as one packed bf16 pair (bf16 rows)
  auto pair_bf = [](const uint4 (&raw)[8], int p, int q) -> uint32_t {
    const uint32_t a = (q < 2) ? raw[2 * p].x : raw[2 * p].y, b = (q < 2) ? raw[2 * p + 1].x : raw[2 * p + 1].y;
    return (q & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
  };
  auto value = [](const uint4 (&raw)[8], int e, int q, bool split) -> float {
    if (split) return __uint_as_float(q == 0 ? raw[e].x : q == 1 ? raw[e].y : q == 2 ? raw[e].z : raw[e].w);
    const uint32_t x = (q < 2) ? raw[e].x : raw[e].y;
    return (q & 1) ? __uint_as_float(x & 0xFFFF0000u) : __uint_as_float(x << 16);
  };
  float bsum[4] = {0.f, 0.f, 0.f, 0.f};
  // the raw rows -> fragments in LDS (and, for B, the column sums)
  auto park = [&](const uint4 (&raw)[8]) {
    if (sb) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int e = 0; e < 8; ++e) bsum[q] += value(raw, e, q, kSplitB);
        if constexpr (kSplitB) {
          uint32_t wv[3][4];
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            uint32_t part[3];
            split_bf3(value(raw, 2 * p, q, true), value(raw, 2 * p + 1, q, true), part);
#pragma unroll
            for (int k = 0; k < 3; ++k) wv[k][p] = part[k];
          }
#pragma unroll
          for (int k = 0; k < 3; ++k) fb[k][sg][swz(sf + q)] = uint4{wv[k][0], wv[k][1], wv[k][2], wv[k][3]};
        } else {
          fb[0][sg][swz(sf + q)] = uint4{pair_bf(raw, 0, q), pair_bf(raw, 1, q), pair_bf(raw, 2, q), pair_bf(raw, 3, q)};
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (kSplitA) {
          uint32_t wv[3][4];
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            uint32_t part[3];
            split_bf3(value(raw, 2 * p, q, true), value(raw, 2 * p + 1, q, true), part);
#pragma unroll
            for (int k = 0; k < 3; ++k) wv[k][p] = part[k];
          }
#pragma unroll
          for (int k = 0; k < 3; ++k) fa[k][sg][swz(sf + q)] = uint4{wv[k][0], wv[k][1], wv[k][2], wv[k][3]};
        } else {
          fa[0][sg][swz(sf + q)] = uint4{pair_bf(raw, 0, q), pair_bf(raw, 1, q), pair_bf(raw, 2, q), pair_bf(raw, 3, q)};
        }
      }
    }
  };
  const int qi = w >> 1, qj = w & 1;
  f32x4 acc[4][4];
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int bj = 0; bj < 4; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};
  constexpr int NJ = 4;  // column blocks whose B fragments are held at a time
  auto compute = [&]() {
#pragma unroll
    for (int j0 = 0; j0 < 4; j0 += NJ) {
      uint4 bq[NJ][PB];
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj)
#pragma unroll
        for (int p = 0; p < PB; ++p) bq[jj][p] = fb[p][g][swz(64 * qj + 16 * (j0 + jj) + c)];
#pragma unroll
      for (int bi = 0; bi < 4; ++bi) {
        uint4 aq[PA];
#pragma unroll
        for (int p = 0; p < PA; ++p) aq[p] = fa[p][g][swz(64 * qi + 16 * bi + c)];
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
#pragma unroll
          for (int ord = 2; ord >= 0; --ord)
#pragma unroll
            for (int pa = 0; pa < PA; ++pa) {
              const int pb = ord - pa;
              if (pb >= 0 && pb < PB) acc[bi][j0 + jj] = mfma_bf16(aq[pa], bq[jj][pb], acc[bi][j0 + jj]);
            }
        }
      }
    }
  };
  int64_t k0 = k_beg;
  keys(k0);
  fetch(k0, rawa);
  keys(k0 + S);
  for (;;) {
    park(rawa);
    lds_barrier();
    const bool more = k0 + S < k_end;
    if (more) {
      fetch(k0 + S, rawa);  // the next step's rows arrive while the waves multiply
      keys(k0 + 2 * S);
    }
    compute();
    lds_barrier();
    if (!more) break;
    k0 += S;
  }
  float* out = partial + chunk * (int64_t)D * D;
#pragma unroll
  for (int bi = 0; bi < 4; ++bi)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t i = TT * ti + 64 * qi + 16 * bi + 4 * g + v;
#pragma unroll
      for (int bj = 0; bj < 4; ++bj) out[i * D + TT * tj + 64 * qj + 16 * bj + c] = acc[bi][bj][v];
    }
  if (colsum && ti == 0) {
    if (sb) {
#pragma unroll
      for (int q = 0; q < 4; ++q) cred[sg][sf + q] = bsum[q];
    }
    __syncthreads();
    if (tid < TT) colsum[chunk * D + TT * tj + tid] = ((cred[0][tid] + cred[1][tid]) + cred[2][tid]) + cred[3][tid];
  }
}

// Chunking of a K-reduction of n rows (deterministic in n): at most
// kSplitPerCu chunks per compute unit, one resident block each.
constexpr int kSplitPerCu = 2;
inline int64_t splitk_chunk(int64_t n) {
  int64_t chunks = cdiv(n, 512);
  const int64_t cap = (int64_t)num_cus() * kSplitPerCu;
  if (chunks > cap) chunks = cap;
  if (chunks < 1) chunks = 1;
  int64_t kc = cdiv(n, chunks);
  kc = cdiv(kc, 64) * 64;
  return kc > 64 ? kc : 64;
}
inline int64_t splitk_max_chunks() { return (int64_t)num_cus() * kSplitPerCu + kSplitGroups + 1; }

// partial must hold splitk_max_chunks() * D * D floats: the grouped stage
// writes its kSplitGroups rows after the chunk rows.
inline int reduce_partials(const float* partial, int64_t chunks, int64_t n, float* tmp, float* out,
                           int accumulate, hipStream_t s) {
  if (chunks <= 2 * kSplitGroups) {
    HG_LAUNCH("splitk_reduce", k_sum_partials, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, partial,
              chunks, n, out, accumulate);
    return HG_OK;
  }
  const int64_t per = cdiv(chunks, kSplitGroups);
  const int64_t groups = cdiv(chunks, per);
  HG_LAUNCH("splitk_reduce", k_sum_partials_grouped, dim3((unsigned)cdiv(n, 256), (unsigned)groups), dim3(256),
            0, s, partial, chunks, n, per, tmp);
  HG_LAUNCH("splitk_reduce", k_sum_partials, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, (const float*)tmp,
            groups, n, out, accumulate);
  return HG_OK;
}

template <int D, class LA, class LB>
int launch_gemm_tn(const char* name, int64_t n_rows, LA la, LB lb, float* partial, float* colsum,
                   float* out, float* out_colsum, int accumulate, hipStream_t s) {
  if (n_rows <= 0) {
    if (!accumulate) {
      HG_TRY(fill_f32(out, 0.f, (int64_t)D * D, s));
      if (out_colsum) HG_TRY(fill_f32(out_colsum, 0.f, D, s));
    }
    return HG_OK;
  }
  const int64_t kc = splitk_chunk(n_rows);
  const int64_t chunks = cdiv(n_rows, kc);
  const bool list_a = la.map.list != nullptr, list_b = lb.map.list != nullptr;
  float* cs = out_colsum ? colsum : nullptr;
  const dim3 grid(tn_grid(D, chunks));
  if constexpr (IsPlainRows<LA>::value && IsPlainRows<LB>::value) {
    // plain feature rows: the bf16 MFMA kernel
    typedef typename std::remove_cv<typename std::remove_pointer<decltype(la.base)>::type>::type TA_;
    typedef typename std::remove_cv<typename std::remove_pointer<decltype(lb.base)>::type>::type TB_;
#define HG_TN_BF(LA_, LB_)                                                                                 \
  do {                                                                                                     \
    if constexpr (D >= 128 && sizeof(TA_) == sizeof(TB_)) {                                              \
      HG_LAUNCH(name, (k_gemm_tn_lds<D, TA_, TB_, LA_, LB_>), grid, dim3(256), 0, s, n_rows, kc, la, lb, partial, \
                cs);                                                                                       \
    } else {                                                                                               \
      HG_LAUNCH(name, (k_gemm_tn_bf<D, TA_, TB_, LA_, LB_>), grid, dim3(256), 0, s, n_rows, kc, la, lb, partial, \
                cs);                                                                                       \
    }                                                                                                      \
  } while (0)
    if (list_a && list_b) {
      HG_TN_BF(true, true);
    } else if (!list_a && !list_b) {
      HG_TN_BF(false, false);
    } else if (list_a) {
      HG_TN_BF(true, false);
    } else {
      HG_TN_BF(false, true);
    }
#undef HG_TN_BF
  } else if (list_a && list_b) {
    HG_LAUNCH(name, (k_gemm_tn<D, LA, LB, true, true>), grid, dim3(256), 0, s, n_rows, kc, la, lb, partial, cs);
  } else if (!list_a && !list_b) {
    HG_LAUNCH(name, (k_gemm_tn<D, LA, LB, false, false>), grid, dim3(256), 0, s, n_rows, kc, la, lb, partial, cs);
  } else if (list_a) {
    HG_LAUNCH(name, (k_gemm_tn<D, LA, LB, true, false>), grid, dim3(256), 0, s, n_rows, kc, la, lb, partial, cs);
  } else {
    HG_LAUNCH(name, (k_gemm_tn<D, LA, LB, false, true>), grid, dim3(256), 0, s, n_rows, kc, la, lb, partial, cs);
  }
  const int64_t cap = (int64_t)num_cus() * kSplitPerCu + 1;
  HG_TRY(reduce_partials(partial, chunks, (int64_t)D * D, partial + cap * D * D, out, accumulate, s));
  if (out_colsum)
    HG_TRY(reduce_partials(colsum, chunks, (int64_t)D, colsum + cap * D, out_colsum, accumulate, s));
  return HG_OK;
}

}  // namespace hg
