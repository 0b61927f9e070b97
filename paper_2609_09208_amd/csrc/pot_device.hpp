// Device-side helpers shared by the gfx950 kernels of libpotattn.
//
// Wave64 is assumed throughout (CDNA4): a wavefront is 64 lanes and one
// 64-element head vector maps one element per lane.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace potattn {

constexpr int kDim = 64;        // head dimension d
constexpr int kExpMax = 6;      // E for a 3-bit exponent field (Sec. II-A)
constexpr int kZeroField = 7;   // e = E + 1 is the exact zero (Sec. II-A)
constexpr int kQMax = 127;      // symmetric INT8 query
constexpr int kFInt = 7;        // internal head-room: every shift F_int - e >= 1
constexpr int kBlock = 256;     // threads per workgroup (4 waves)
constexpr int kTile = 256;      // keys per tile, one key per thread in scoring

// fp32 log2(e) rounded to nearest, bit pattern 0x3FB8AA3B.
__device__ __forceinline__ float log2e_f32() { return __uint_as_float(0x3FB8AA3Bu); }

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Radix-2 Walsh-Hadamard butterfly over one 64-vector held one element per
// lane, in fp64, stages of span 1, 2, 4, ..., 32 mapping (a, b) to
// (a + b, a - b). For fp16 inputs every partial sum is exact in fp64; for fp32
// inputs this fixed stage order is the rotation's definition.
__device__ __forceinline__ double wave_fwht64(double v) {
  const int lane = lane_id();
#pragma unroll
  for (int h = 1; h < kDim; h <<= 1) {
    double o = __shfl_xor(v, h, 64);
    v = (lane & h) ? (o - v) : (v + o);
  }
  return v;
}

// INT8 quantisation of one 64-vector held one element per lane (Sec. II-A):
// amax = max|x|, step = fl32(amax/127), code = clamp(rne(fl32(x *
// fl32(127/amax))), -127, 127). amax = 0 gives code 0 and step 0.
__device__ __forceinline__ int wave_quantize_int8(float x, float* step) {
  const float amax = wave_max(fabsf(x));
  if (amax == 0.0f) {
    *step = 0.0f;
    return 0;
  }
  const float inv = 127.0f / amax;  // correctly rounded division
  float r = rintf(__fmul_rn(x, inv));
  r = fminf(fmaxf(r, -127.0f), 127.0f);
  *step = amax / 127.0f;  // correctly rounded division
  return (int)r;
}

}  // namespace potattn
