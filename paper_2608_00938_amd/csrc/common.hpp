// Device helpers shared by the gfx950 kernels of the decode-attention library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace grace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
// 16-byte register chunk.  A native vector (not HIP's union-based uint4) so that
// arrays of chunks stay in VGPRs.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

// Storage tags: the element type in memory.  Arithmetic is always fp32.
struct F32 {
  using storage = float;
  static constexpr int kBytes = 4;
};
struct BF16 {
  using storage = uint16_t;
  static constexpr int kBytes = 2;
};

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp32 pair -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 v = {lo, hi};
  bf16x2 b = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, b);
}

// A 16-byte chunk as fp32 lanes: 4 floats or 8 bf16.
template <class T> struct Chunk;
template <> struct Chunk<F32> {
  static constexpr int kElems = 4;
  __device__ __forceinline__ static void unpack(const u32x4& u, float* f) {
    f[0] = __uint_as_float(u.x); f[1] = __uint_as_float(u.y);
    f[2] = __uint_as_float(u.z); f[3] = __uint_as_float(u.w);
  }
  __device__ __forceinline__ static u32x4 pack(const float* f) {
    return u32x4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                 __float_as_uint(f[3])};
  }
};
template <> struct Chunk<BF16> {
  static constexpr int kElems = 8;
  __device__ __forceinline__ static void unpack(const u32x4& u, float* f) {
    f[0] = __uint_as_float(u.x << 16); f[1] = __uint_as_float(u.x & 0xffff0000u);
    f[2] = __uint_as_float(u.y << 16); f[3] = __uint_as_float(u.y & 0xffff0000u);
    f[4] = __uint_as_float(u.z << 16); f[5] = __uint_as_float(u.z & 0xffff0000u);
    f[6] = __uint_as_float(u.w << 16); f[7] = __uint_as_float(u.w & 0xffff0000u);
  }
  __device__ __forceinline__ static u32x4 pack(const float* f) {
    return u32x4{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]),
                 pack_bf16x2(f[4], f[5]), pack_bf16x2(f[6], f[7])};
  }
};

// Sum over aligned groups of G lanes (G in {1,2,4,8,16,32}); every lane of the
// group ends with the group total.  DPP for partners inside a row of 16 lanes,
// a swizzle across the two rows of a 32-lane half.
template <int G>
__device__ __forceinline__ float group_sum(float x) {
  if constexpr (G >= 2)
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                               0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
  if constexpr (G >= 4)
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                               0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
  if constexpr (G >= 8)
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                               0x141, 0xF, 0xF, false));  // row_half_mirror
  if constexpr (G >= 16)
    x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                               0x140, 0xF, 0xF, false));  // row_mirror
  if constexpr (G >= 32)
    x += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, x),
                                                               (16 << 10) | 0x1F));     // xor 16
  return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Unsigned 32-bit division by a divisor fixed for a whole launch (1 <= d <=
// 2^31), as one high multiply, a subtract, an add and two shifts (Granlund and
// Montgomery, "Division by invariant integers using multiplication", PLDI 1994,
// Sec. 4): with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1,
// n / d = (t + ((n - t) >> min(l, 1))) >> max(l - 1, 0) where t = mulhi(m, n).
// The constants are computed on the host.
struct FastDiv {
  uint32_t m = 1, s1 = 0, s2 = 0;
  FastDiv() = default;
  __host__ explicit FastDiv(uint32_t d) {
    uint32_t l = 0;
    while (l < 32 && (1ull << l) < d) ++l;
    m = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
    s1 = l < 1 ? l : 1;
    s2 = l < 1 ? 0 : l - 1;
  }
  __device__ __forceinline__ uint32_t div(uint32_t n) const {
    const uint32_t t = __umulhi(m, n);
    return (t + ((n - t) >> s1)) >> s2;
  }
};

// XCD-aware workgroup order.  Consecutive workgroup ids go round-robin over
// the 8 XCDs; the remapped index i' gives XCD x the contiguous range
// [x*n/8, (x+1)*n/8), processed in order, so that work items that share data
// (the beam tiles of one request and head, or the beam rows of one request)
// run on one XCD and close in time, and that XCD's L2 serves them all.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t i, uint32_t n) {
  constexpr uint32_t kXcds = 8;
  if (n % kXcds != 0) return i;
  return (i % kXcds) * (n / kXcds) + i / kXcds;
}

}  // namespace grace
