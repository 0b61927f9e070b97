// Device-side helpers shared by the gfx950 kernels of libpotattn.
//
// Wave64 is assumed throughout (CDNA4): a wavefront is 64 lanes and one
// 64-element head vector maps one element per lane.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pot_launch.hpp"

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

// One DPP lane move inside each row of 16 lanes (bound_ctrl: every source
// lane exists for the patterns used here).
template <int kCtrl>
__device__ __forceinline__ float dpp_move(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), kCtrl,
                                                            0xF, 0xF, true));
}

// Maximum over the wave (fmaxf: NaN ignored unless every lane is NaN), with
// register-to-register moves only: neighbour and pair swaps, the mirror
// inside each half row and each row (DPP), then the swaps of rows 0-1 / 2-3
// and of the two halves (v_permlane16_swap, v_permlane32_swap). A maximum
// does not care which lane of the other group it meets.
__device__ __forceinline__ float wave_max(float v) {
  constexpr int kQuadSwap1 = 0xB1, kQuadSwap2 = 0x4E, kRowHalfMirror = 0x141, kRowMirror = 0x140;
  v = fmaxf(v, dpp_move<kQuadSwap1>(v));
  v = fmaxf(v, dpp_move<kQuadSwap2>(v));
  v = fmaxf(v, dpp_move<kRowHalfMirror>(v));
  v = fmaxf(v, dpp_move<kRowMirror>(v));
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
  v = fmaxf(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
  return fmaxf(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
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

// Log-nearest PoT-Mk code of one element, mantissa width K (Sec. II-A, eq.
// pot; Sec. II-D, eq. mant), from u = RN(|x| / s) (a zero or NaN x gives a
// ratio at or below the zero cut, or NaN); s_bad: s is not positive. Branch-
// free. Returns the nibble (neg<<3 | e, or 7 for zero) and the mantissa j.
template <int K>
__device__ __forceinline__ int code_from_ratio(float u, bool neg, bool s_bad,
                                               const EncodeTables& tab, int* j_out) {
  constexpr int n = 1 << K;
  const bool zero = s_bad || !(u > tab.zero_cut);  // also a NaN ratio
  const uint32_t ub = __float_as_uint(u);
  const int e2 = (int)(ub >> 23) - 127;  // u > 2^-7 (normal) where it matters
  const float m = __uint_as_float((ub & 0x007FFFFFu) | 0x3F800000u);  // [1, 2)
  if constexpr (K == 0) {
    // above the cut m rounds up into the next binade; u >= 1 saturates at
    // e = 0; below 2^-E (above the zero cut) the smallest magnitude
    const int c = (m > tab.cut[0]) ? 1 : 0;
    const int e = min(max(-e2 - c, 0), kExpMax);
    *j_out = 0;
    return zero ? kZeroField : ((neg ? 8 : 0) | e);
  } else {
    int c = 0;
#pragma unroll
    for (int i = 0; i < n; ++i) c += (m > tab.cut[i]) ? 1 : 0;
    // c == n rounds up to the next binade's first value; u >= 1 is the top
    // binade, saturating at its largest value; below 2^-E (above the zero
    // cut) the smallest magnitude
    int e = (c == n) ? -e2 - 1 : -e2;
    int j = (c == n) ? 0 : c;
    e = (e2 >= 0) ? 0 : e;
    j = (e2 > 0) ? n - 1 : ((e2 == 0) ? min(c, n - 1) : j);
    j = (e > kExpMax) ? 0 : j;
    e = min(e, kExpMax);
    *j_out = zero ? 0 : j;
    return zero ? kZeroField : ((neg ? 8 : 0) | e);
  }
}

// The same from x and the row scale s (one correctly rounded division).
template <int K>
__device__ __forceinline__ int classify(float x, float s, const EncodeTables& tab, int* j_out) {
  return code_from_ratio<K>(fabsf(x) / s, x < 0.0f, !(s > 0.0f), tab, j_out);
}

// Encodes one 64-element fp16 key row with the calling wave, one element per
// lane (Sec. II-A, II-D): optional exact fp64 Walsh-Hadamard rotation, the row
// scale (scale_mode 0: s = max|K'| written to *scale; 1: s read from *scale),
// the log-nearest code of every element, sign/exponent nibbles packed by lane
// shuffles (element m at bit 4*(m%8) of dword m/8 of se_out) and mantissa
// bit-planes by ballots (bit m of the 64-bit plane b of m_out is bit b of j_m).
template <int K>
__device__ __forceinline__ void encode_key_row_wave(const __half* __restrict__ k_row,
                                                    int hadamard, int scale_mode,
                                                    float* __restrict__ scale,
                                                    uint8_t* __restrict__ se_out,
                                                    uint8_t* __restrict__ m_out,
                                                    const EncodeTables& tab) {
  const int lane = lane_id();
  float x = __half2float(k_row[lane]);
  if (hadamard) x = (float)(wave_fwht64((double)x) * 0.125);
  float s;
  if (scale_mode == 0) {
    s = wave_max(fabsf(x));
    if (lane == 0) *scale = s;
  } else {
    s = *scale;
  }
  int j;
  const int nib = classify<K>(x, s, tab, &j);
  uint32_t w = (uint32_t)nib << (4 * (lane & 7));
  w |= __shfl_xor(w, 1, 64);
  w |= __shfl_xor(w, 2, 64);
  w |= __shfl_xor(w, 4, 64);
  if ((lane & 7) == 0) reinterpret_cast<uint32_t*>(se_out)[lane >> 3] = w;
#pragma unroll
  for (int b = 0; b < K; ++b) {
    const unsigned long long plane = __ballot((j >> b) & 1);
    if (lane == 0) reinterpret_cast<unsigned long long*>(m_out)[b] = plane;
  }
}

// Value cache layout: token t of a sequence, dim d, lives at
// ((t/8)*8) * 64 + d * 8 + t % 8 halves from the sequence's base. Stores one
// token's 64 fp16 values with the calling wave (lane = dim).
__device__ __forceinline__ void store_value_token_wave(const uint16_t* __restrict__ v_row,
                                                       uint16_t* __restrict__ v_seq,
                                                       int64_t t) {
  const int lane = lane_id();
  v_seq[(t / 8) * 8 * kDim + lane * 8 + t % 8] = v_row[lane];
}

// INT8 values with a power-of-two per-token scale (Sec. II-E) for one token,
// quantised and stored by the calling wave (lane = dim): g is the largest
// integer with max|v| 2^g <= 127 (0 for an all-zero row) and v^ = rne(v 2^g),
// so |v^| <= 127. The byte cache holds v^ + 128 (offset binary) at the
// token-interleaved position ((t/8)*8) * 64 + d * 8 + t % 8 of the sequence,
// and exp_seq[t] = g; the value is v^ 2^-g.
__device__ __forceinline__ void store_value_token_i8_wave(const uint16_t* __restrict__ v_row,
                                                          uint8_t* __restrict__ v_seq,
                                                          int8_t* __restrict__ exp_seq,
                                                          int64_t t) {
  const int lane = lane_id();
  const float v = __half2float(__ushort_as_half(v_row[lane]));
  const float amax = wave_max(fabsf(v));
  int g = 0;
  if (amax > 0.0f) {
    // amax in [2^e, 2^(e+1)) with e = frexp exponent - 1, so amax 2^(6-e) is
    // in [64, 128) (exact power-of-two scaling)
    const int e = __builtin_amdgcn_frexp_expf(amax) - 1;
    g = (__builtin_amdgcn_ldexpf(amax, 6 - e) <= 127.0f) ? 6 - e : 5 - e;
  }
  const int c = (int)rintf(__builtin_amdgcn_ldexpf(v, g));
  v_seq[(t / 8) * 8 * kDim + lane * 8 + t % 8] = (uint8_t)(c + 128);
  if (lane == 0) exp_seq[t] = (int8_t)g;
}

}  // namespace potattn
