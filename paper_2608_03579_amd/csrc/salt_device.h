// Device-side element helpers of libsalt (gfx950): bf16 / fp32 vectors of 8
// elements, conversions with round-to-nearest-even, dot products and the MFMA
// steps the kernels use.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace salt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest even: gfx950's packed conversion
// (v_cvt_pk_bf16_f32), two values per instruction; `lo` lands in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

// ---- buffer resources ----------------------------------------------------------
// A raw buffer resource (base, size in bytes) and 32-bit byte offsets into it.
// The hardware range check makes an access at an offset >= the size read zero
// and discards a store, so a lane with nothing to load or store is given the
// offset kOob: no branch, no clamp, and every lane issues the same memory
// instructions (the compiler's counts of outstanding loads stay exact).  Every
// access a kernel makes is either wholly inside its buffer or at kOob; the
// host keeps every buffer below 2^31 bytes.
typedef __amdgpu_buffer_rsrc_t Rsrc;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr uint32_t kOob = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;      // raw 32-bit dword access, no swizzle (gfx9 family)

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}
__device__ __forceinline__ uint4 buf_load16(Rsrc r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void buf_store16(Rsrc r, uint32_t off, uint4 v) {
  const u32x4 w = {v.x, v.y, v.z, v.w};
  __builtin_amdgcn_raw_buffer_store_b128(w, r, (int)off, 0, 0);
}
__device__ __forceinline__ float buf_load_f32(Rsrc r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
}
__device__ __forceinline__ void buf_store_f32(Rsrc r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, 0, 0);
}
__device__ __forceinline__ float4 buf_load_f32x4(Rsrc r, uint32_t off) {
  const uint4 v = buf_load16(r, off);
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
}
__device__ __forceinline__ float4 f4_add(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}
// `off` if `ok`, else the out-of-range offset
__device__ __forceinline__ uint32_t oob_unless(bool ok, uint32_t off) { return ok ? off : kOob; }

template <typename E>
struct Ops;

// bf16 storage (uint16 bit patterns); a vector is 8 elements in one uint4.
template <>
struct Ops<uint16_t> {
  using Vec = uint4;
  static __device__ __forceinline__ Vec zero() { return make_uint4(0u, 0u, 0u, 0u); }
  static __device__ __forceinline__ Vec load(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  static __device__ __forceinline__ Vec bload(Rsrc r, uint32_t off) { return buf_load16(r, off); }
  static __device__ __forceinline__ void bstore(Rsrc r, uint32_t off, const float* f) {
    buf_store16(r, off, make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                                   pack_bf16x2(f[6], f[7])));
  }
  static __device__ __forceinline__ void to_f32(const Vec& v, float* o) {
    o[0] = bf_lo(v.x); o[1] = bf_hi(v.x); o[2] = bf_lo(v.y); o[3] = bf_hi(v.y);
    o[4] = bf_lo(v.z); o[5] = bf_hi(v.z); o[6] = bf_lo(v.w); o[7] = bf_hi(v.w);
  }
  static __device__ __forceinline__ void store(uint16_t* p, const float* f) {
    uint4 w;
    w.x = pack_bf16x2(f[0], f[1]);
    w.y = pack_bf16x2(f[2], f[3]);
    w.z = pack_bf16x2(f[4], f[5]);
    w.w = pack_bf16x2(f[6], f[7]);
    *reinterpret_cast<uint4*>(p) = w;
  }
  // acc + sum_e a[e] * b[e]; bf16 products are exact in fp32
  static __device__ __forceinline__ float dot(const Vec& a, const Vec& b, float acc) {
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.x), __builtin_bit_cast(bf16x2, b.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.y), __builtin_bit_cast(bf16x2, b.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.z), __builtin_bit_cast(bf16x2, b.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a.w), __builtin_bit_cast(bf16x2, b.w), acc, false);
    return acc;
  }
  // One 16x16x32 step: lane l brings row (l & 15) of the left operand and
  // column (l & 15) of the right one, 8 consecutive k each (k = 8 (l >> 4) ..);
  // lane l receives column (l & 15), rows 4 (l >> 4) .. + 3 of the product.
  static __device__ __forceinline__ f32x4 mma(const Vec& a, const Vec& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
};

// fp32 storage; a vector is 8 elements in two float4.
template <>
struct Ops<float> {
  struct Vec {
    float4 lo, hi;
  };
  static __device__ __forceinline__ Vec zero() {
    return Vec{make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
  }
  static __device__ __forceinline__ Vec load(const float* p) {
    return Vec{*reinterpret_cast<const float4*>(p), *reinterpret_cast<const float4*>(p + 4)};
  }
  // (kOob + 16 is still out of range)
  static __device__ __forceinline__ Vec bload(Rsrc r, uint32_t off) {
    const uint4 a = buf_load16(r, off), b = buf_load16(r, off + 16);
    return Vec{make_float4(__uint_as_float(a.x), __uint_as_float(a.y), __uint_as_float(a.z), __uint_as_float(a.w)),
               make_float4(__uint_as_float(b.x), __uint_as_float(b.y), __uint_as_float(b.z), __uint_as_float(b.w))};
  }
  static __device__ __forceinline__ void bstore(Rsrc r, uint32_t off, const float* f) {
    buf_store16(r, off, make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                                   __float_as_uint(f[3])));
    buf_store16(r, off + 16, make_uint4(__float_as_uint(f[4]), __float_as_uint(f[5]), __float_as_uint(f[6]),
                                        __float_as_uint(f[7])));
  }
  static __device__ __forceinline__ void to_f32(const Vec& v, float* o) {
    o[0] = v.lo.x; o[1] = v.lo.y; o[2] = v.lo.z; o[3] = v.lo.w;
    o[4] = v.hi.x; o[5] = v.hi.y; o[6] = v.hi.z; o[7] = v.hi.w;
  }
  static __device__ __forceinline__ void store(float* p, const float* f) {
    *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
  }
  static __device__ __forceinline__ float dot(const Vec& a, const Vec& b, float acc) {
    float x[8], y[8];
    to_f32(a, x);
    to_f32(b, y);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf(x[e], y[e], acc);
    return acc;
  }
  // Eight 16x16x4 fp32 steps: in step e, lane group g = l >> 4 supplies k = 8g + e,
  // so the eight steps together cover the same 32 k as one bf16 step.
  static __device__ __forceinline__ f32x4 mma(const Vec& a, const Vec& b, f32x4 c) {
    float x[8], y[8];
    to_f32(a, x);
    to_f32(b, y);
#pragma unroll
    for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[e], y[e], c, 0, 0, 0);
    return c;
  }
};

}  // namespace salt
