// Scalar arithmetic shared by the GEMM epilogues and the reduction: bf16
// conversion (round to nearest even) and the exact-erf GeLU with its
// derivative (Sec. 2.1).  One definition, so a fused GEMM + peer-sum
// epilogue and a separate reduction of the same partials give the same bits.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace atp {
namespace epi {

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0x7fc0u;  // NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ float gelu_f(float x) {
    return 0.5f * x * (1.0f + erff(x * 0.70710678118654752440f));
}

__device__ __forceinline__ float gelu_grad_f(float x) {
    const float cdf = 0.5f * (1.0f + erff(x * 0.70710678118654752440f));
    const float pdf = 0.39894228040143267794f * expf(-0.5f * x * x);
    return cdf + x * pdf;
}

}  // namespace epi
}  // namespace atp
