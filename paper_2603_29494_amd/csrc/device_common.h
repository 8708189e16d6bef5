// Device-side helpers shared by the HIP kernels of libvecattn (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vecattn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp64 -> bf16 bit pattern, round to nearest, ties to even, one rounding step.
// Normal results: round the 52-bit double mantissa to 7 bits at bit 45 with
// integer arithmetic (a carry into the exponent is the correct renormalisation).
// Results below 2^-126 land on bf16's subnormal grid of spacing 2^-133.
__device__ __forceinline__ uint16_t f64_to_bf16_rne(double x) {
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  const uint16_t sign = static_cast<uint16_t>((u >> 48) & 0x8000u);
  const uint64_t a = u & 0x7FFFFFFFFFFFFFFFull;
  if (a >= 0x7FF0000000000000ull) return a > 0x7FF0000000000000ull ? 0x7FC0 : (sign | 0x7F80);
  const int e = static_cast<int>(a >> 52) - 1023;
  if (e < -126) {
    const double r = __builtin_rint(__builtin_fabs(x) * 0x1p133);  // exact scale, RNE
    return sign | static_cast<uint16_t>(r);
  }
  const uint64_t lsb = (a >> 45) & 1u;
  const uint64_t t = (a + 0x00000FFFFFFFFFFFull + lsb) >> 45;  // half-ulp minus one, plus lsb
  const int ef = static_cast<int>(t >> 7) - 1023 + 127;
  if (ef >= 255) return sign | 0x7F80;
  return sign | static_cast<uint16_t>((ef << 7) | (t & 0x7F));
}

// XCD-aware work order: the hardware hands workgroup x to XCD x % 8; item
// (x % 8) * per + x / 8 gives each XCD a contiguous range of work items, so
// the items of one head share that XCD's L2.
__device__ __forceinline__ int64_t xcd_work_item(int64_t per_xcd) {
  const int64_t x = blockIdx.x;
  return (x & 7) * per_xcd + (x >> 3);
}

__device__ __forceinline__ float wave_max_xor32(float x) {
  return fmaxf(x, __shfl_xor(x, 32));
}

}  // namespace vecattn
