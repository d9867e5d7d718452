// Device helpers shared by the gfx950 kernels of libwtconv (storage-type
// conversion and the Haar butterfly). Internal; not part of the public ABI.
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace wtc {

#define DEV __device__ __forceinline__

// ----------------------------------------------------------------------------
// storage types: float32, bfloat16 (as uint16_t bits) and IEEE half
// ----------------------------------------------------------------------------
DEV float to_f32(float v) { return v; }
DEV float to_f32(uint16_t v) { return __uint_as_float(((uint32_t)v) << 16); }  // bf16
DEV float to_f32(_Float16 v) { return (float)v; }

template <typename T>
DEV T from_f32(float v);
template <>
DEV float from_f32<float>(float v) { return v; }
template <>
DEV uint16_t from_f32<uint16_t>(float v)  // bf16, round to nearest even
{
    // gfx950 converts in one instruction (v_cvt_pk_bf16_f32, round to nearest
    // even, NaN stays NaN); measured bit-identical to the integer rounding
    // (add 0x7fff plus the lowest kept bit, truncate) on 2^24 inputs including
    // ties, subnormals and infinities.
    return __builtin_bit_cast(uint16_t, (__bf16)v);
}
template <>
DEV _Float16 from_f32<_Float16>(float v) { return (_Float16)v; }

// Unnormalised Haar butterfly of the 2x2 patch [[a, b], [c, d]]:
// (LL, LH, HL, HH) = (a+b+c+d, a+b-c-d, a-b+c-d, a-b-c+d), eq. (butterfly)
// without its factor 1/2.
DEV void butterfly(float a, float b, float c, float d, float (&o)[4])
{
    const float ab = a + b, cd = c + d, amb = a - b, cmd = c - d;
    o[0] = ab + cd;
    o[1] = ab - cd;
    o[2] = amb + cmd;
    o[3] = amb - cmd;
}

}  // namespace wtc
