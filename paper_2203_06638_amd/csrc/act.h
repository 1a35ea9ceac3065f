// act.h -- storage types of activations and the conversions between them.
//
// Activations and activation gradients are stored either as float32 or as
// bfloat16 (the upper 16 bits of a float32; conversion from float32 rounds to
// nearest, ties to even).  Kernels compute in float32 either way; these
// overloads load and store channel quads (4 consecutive NHWC elements) and
// single elements in either type.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace lpp {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16;   // bfloat16 bit pattern

__device__ __forceinline__ bf16 to_bf16(float x) { return __builtin_bit_cast(bf16, (__bf16)x); }
__device__ __forceinline__ float from_bf16(bf16 h) { return __uint_as_float((uint32_t)h << 16); }
// two values packed low | high << 16
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)to_bf16(lo) | ((uint32_t)to_bf16(hi) << 16);
}

__device__ __forceinline__ f4 ld4(const float* p, long q) { return ((const f4*)p)[q]; }
__device__ __forceinline__ f4 ld4(const bf16* p, long q) {
    const uint2 u = ((const uint2*)p)[q];
    return f4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
              __uint_as_float(u.y & 0xffff0000u)};
}
__device__ __forceinline__ void st4(float* p, long q, f4 v) { ((f4*)p)[q] = v; }
__device__ __forceinline__ void st4(bf16* p, long q, f4 v) {
    ((uint2*)p)[q] = uint2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
}
// 16 bytes of storage-type values (4 floats or 8 bf16) from floats, one store
__device__ __forceinline__ void st16(float* p, const float* v) { *(f4*)p = f4{v[0], v[1], v[2], v[3]}; }
__device__ __forceinline__ void st16(bf16* p, const float* v) {
    *(uint4*)p = uint4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                       pack_bf16x2(v[6], v[7])};
}
__device__ __forceinline__ float ld1(const float* p, long i) { return p[i]; }
__device__ __forceinline__ float ld1(const bf16* p, long i) { return from_bf16(p[i]); }
__device__ __forceinline__ void st1(float* p, long i, float v) { p[i] = v; }
__device__ __forceinline__ void st1(bf16* p, long i, float v) { p[i] = to_bf16(v); }

}  // namespace lpp
