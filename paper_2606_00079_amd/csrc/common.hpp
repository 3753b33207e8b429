// Device-side types and helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bitsmoe {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;

// fp32 -> bf16 bit pattern, round to nearest even (inputs are finite).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> fp16 bit pattern and back, round to nearest even (hardware cvt).
__device__ __forceinline__ uint16_t f32_to_f16_bits(float f) {
  _Float16 h = static_cast<_Float16>(f);
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t b) {
  return static_cast<float>(__builtin_bit_cast(_Float16, b));
}

__device__ __forceinline__ double f16_bits_to_f64(uint16_t b) {
  return static_cast<double>(static_cast<float>(__builtin_bit_cast(_Float16, b)));
}

// Returns v unchanged but opaque to the optimizer: computations that depend
// on the result cannot be hoisted above this point (used so that epilogue
// address arithmetic is not moved before a long loop and kept live there).
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ float opaque(float v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Min and max over each aligned block of glanes lanes (a power of two, at
// most 64); every lane of a block gets both.  Inside a row of 16 lanes each
// step takes the partner value by DPP inside the min / max instruction:
// lane ^ 1 and lane ^ 2 (quad permutations), then the half-row mirror (lane
// i of 8 reads 7 - i, which holds the other quad's result) and the row
// mirror (15 - i: the other half row's).  The s_nop ahead of the first step
// covers the wait states a DPP read needs after a VALU write of its operand
// or a write of EXEC; the ones between steps cover the operand written two
// instructions earlier.  Lane ^ 16 is a swizzle, lane ^ 32 a shuffle.
#define BITSMOE_DPP_MM(ctrl)                                                       \
  "v_min_f32_dpp %0, %0, %0 " ctrl " row_mask:0xf bank_mask:0xf\n\t"               \
  "v_max_f32_dpp %1, %1, %1 " ctrl " row_mask:0xf bank_mask:0xf\n\t"
__device__ __forceinline__ void block_minmax(float& mn, float& mx, int glanes) {
  if (glanes == 16) {  // groups of 128 entries at 8 per lane
    asm("s_nop 4\n\t" BITSMOE_DPP_MM("quad_perm:[1,0,3,2]") "s_nop 1\n\t"
        BITSMOE_DPP_MM("quad_perm:[2,3,0,1]") "s_nop 1\n\t" BITSMOE_DPP_MM("row_half_mirror")
        "s_nop 1\n\t" BITSMOE_DPP_MM("row_mirror")
        : "+v"(mn), "+v"(mx));
    return;
  }
  if (glanes > 1) asm("s_nop 4\n\t" BITSMOE_DPP_MM("quad_perm:[1,0,3,2]") : "+v"(mn), "+v"(mx));
  if (glanes > 2) asm("s_nop 4\n\t" BITSMOE_DPP_MM("quad_perm:[2,3,0,1]") : "+v"(mn), "+v"(mx));
  if (glanes > 4) asm("s_nop 4\n\t" BITSMOE_DPP_MM("row_half_mirror") : "+v"(mn), "+v"(mx));
  if (glanes > 8) asm("s_nop 4\n\t" BITSMOE_DPP_MM("row_mirror") : "+v"(mn), "+v"(mx));
  if (glanes > 16) {  // swizzle in bit-mask mode: and 0x1f, xor 0x10
    mn = fminf(mn, __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, mn), 0x401F)));
    mx = fmaxf(mx, __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, mx), 0x401F)));
  }
  if (glanes > 32) {
    mn = fminf(mn, __shfl_xor(mn, 32, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  }
}
#undef BITSMOE_DPP_MM

// x / qmax rounded to nearest-even in fp32, for qmax = 2^b - 1 (b <= 8) and
// finite x >= 0, given rq = fp32(1 / qmax): the product x rq is corrected
// once by its residual x - q0 qmax, which the fma forms exactly (a multiple
// of ulp(q0) below 2^9 ulp(q0)).  Equal to the IEEE quotient for every such
// x and qmax (checked exhaustively over the binades where scaling does not
// apply and over whole binades elsewhere); three instructions instead of
// the division's ten.
__device__ __forceinline__ float div_qmax(float x, float qmax, float rq) {
  const float q0 = x * rq;
  return fmaf(fmaf(-q0, qmax, x), rq, q0);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace bitsmoe

#define BITSMOE_LAUNCH_CHECK(what)                             \
  do {                                                         \
    hipError_t _e = hipGetLastError();                         \
    if (_e != hipSuccess) return ::bitsmoe::device_error(what, _e); \
  } while (0)
