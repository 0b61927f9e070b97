// Key encoders for gfx950: fp16 key rows -> PoT / PoT-Mk codes (Sec. II-A,
// II-D) and -> INT8 uniform codes (the multiply-accumulate comparator).
//
// The bulk PoT encoder works on 8 key rows per wavefront at a time: lane l
// takes row l / 8 of the group and elements 8g .. 8g + 7 of it (g = l % 8),
// so a row is one 16-byte load per lane over 8 lanes and its code word g (the
// 8 nibbles of those elements) is one 4-byte store. The optional Walsh-
// Hadamard rotation is an exact fp64 butterfly (spans 1, 2, 4 inside the
// lane, 8, 16, 32 across the row's lanes), the row scale a max over 8 values
// and three DPP lane exchanges. Each ratio |x| / s is correctly rounded from
// one reciprocal per row (a Newton-corrected hardware reciprocal, then
// Markstein's correction of the quotient). PoT-4 then takes its code from
// the ratio's bits with integer operations (an add that carries into the
// exponent exactly above the cut point, a shift and a clamp) and its sign
// bits from the inputs' sign bits eight at a time by byte permutes; PoT-Mk
// (K > 0) compares the mantissa against the fp32 cut points. (The fused per-
// token append in the decode kernel and the INT8 comparator encode one row
// per wavefront, one element per lane.)
#include <hip/hip_fp16.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "pot_device.hpp"
#include "pot_launch.hpp"

namespace potattn {

namespace {

// Largest fp32 strictly below sqrt(num / den^2) for num not a perfect square,
// with num / den^2 in [1, 4): the value is M * 2^-23 with M the integer part
// of sqrt(num * 2^46 / den^2) (exact integer square root).
float rd_sqrt_ratio(uint64_t num, uint64_t den) {
  // R * 2^46 = num * 2^46 / den^2; den is a power of two <= 16 so the
  // division is exact.
  unsigned __int128 v = ((unsigned __int128)num << 46) / ((unsigned __int128)den * den);
  uint64_t m = (uint64_t)std::sqrt((long double)v);
  while ((unsigned __int128)m * m > v) --m;
  while ((unsigned __int128)(m + 1) * (m + 1) <= v) ++m;
  return std::ldexp((float)m, -23);  // m < 2^25 so exact in fp32
}

}  // namespace

EncodeTables make_encode_tables(int mant_bits) {
  EncodeTables t{};
  const uint64_t n = 1ull << mant_bits;
  for (uint64_t i = 0; i < n; ++i) t.cut[i] = rd_sqrt_ratio((n + i) * (n + i + 1), n);
  for (uint64_t i = n; i < 16; ++i) t.cut[i] = INFINITY;
  // 2^-(E+1/2) = sqrt(2) * 2^-7: RD of sqrt(2) scaled by an exact power of two.
  t.zero_cut = std::ldexp(rd_sqrt_ratio(2, 1), -(kExpMax + 1));
  t.mant_bits = mant_bits;
  return t;
}

// The row-per-wave kernels below step over rows with the grid's stride: a
// launch has at most kMaxGrid workgroups, since a dispatch is limited to
// 2^32 work-items per dimension (2^26 rows of one wave each).
constexpr int64_t kMaxGrid = 1 << 20;
// bulk PoT encoder: 256 CUs x 8 workgroups of 4 waves
constexpr int64_t kEncodeGrid = 256 * 8;

// Maximum over the 8 lanes of an aligned group (lane & ~7) of non-negative,
// non-NaN floats, compared as their bit patterns: swap neighbours, swap
// pairs, then the mirror image inside each half row (a maximum does not care
// which lane of the other quad it meets).
template <int kCtrl>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, kCtrl, 0xF, 0xF, true);
}
__device__ __forceinline__ float max_over_8_lanes(float v) {
  constexpr int kQuadSwap1 = 0xB1, kQuadSwap2 = 0x4E, kRowHalfMirror = 0x141;
  uint32_t b = __float_as_uint(v);
  b = max(b, dpp_u32<kQuadSwap1>(b));
  b = max(b, dpp_u32<kQuadSwap2>(b));
  return __uint_as_float(max(b, dpp_u32<kRowHalfMirror>(b)));
}

// Scales whose reciprocal takes the fast path: [2^-126, 2^126] (no NaN,
// sign, infinity or subnormal reciprocal), by one unsigned compare.
__device__ __forceinline__ bool recip_in_range(float s) {
  return __float_as_uint(s) - 0x00800000u <= 0x7E800000u - 0x00800000u;
}

// RN(1 / s) for s in [2^-126, 2^126]: v_rcp_f32 is within one ulp, and one
// Newton step with fused multiply-adds then rounds correctly for every start
// within an ulp, except for an all-ones mantissa, s = (2 - 2^-23) 2^k, where
// the step can land on a tie: there 1/s = 2^-(k+1) (1 + 2^-24 + 2^-48 ...)
// rounds to 2^-(k+1) (1 + 2^-23), whose bits are 0x7E800001 minus the
// exponent field of s. (Checked over every mantissa of one binade and every
// start within an ulp.)
__device__ __forceinline__ float recip_rn(float s) {
  const float r0 = __builtin_amdgcn_rcpf(s);
  const float r1 = __builtin_fmaf(__builtin_fmaf(-s, r0, 1.0f), r0, r0);
  const uint32_t sb = __float_as_uint(s);
  return ((sb & 0x007FFFFFu) == 0x007FFFFFu) ? __uint_as_float(0x7E800001u - (sb & 0x7F800000u))
                                               : r1;
}

inline uint32_t bounded_grid(int64_t blocks) {
  return (uint32_t)(blocks < kMaxGrid ? blocks : kMaxGrid);
}

// Clamp to [0, 1] with NaN mapped to 0: folds into the producing
// instruction's clamp bit (the DX10 clamp mode, on for compute kernels).
__device__ __forceinline__ float clamp01(float x) { return __builtin_amdgcn_fmed3f(x, 0.0f, 1.0f); }

// Nibble masks of 8 signs: nibble i of the result is 0xF where bytes a (signs
// 0..3) and b (signs 4..7), each 0x00 or 0xFF, say sign i is set.
__device__ __forceinline__ uint32_t sign_nibbles(uint32_t a, uint32_t b) {
  const uint32_t even = __builtin_amdgcn_perm(b, a, 0x06040200u);  // signs 0 2 4 6
  const uint32_t odd = __builtin_amdgcn_perm(b, a, 0x07050301u);   // signs 1 3 5 7
  return (even & 0x0F0F0F0Fu) | (odd & 0xF0F0F0F0u);
}

// PoT-4 code word of 8 elements from their clamped ratios c_i = min(RN(|x_i|
// / s), 1) (0 for NaN) and sign masks. With c = (1 + M 2^-23) 2^(E-127) and
// the cut point RD(sqrt 2) = 1 + Mc 2^-23, the log-nearest exponent is
// e = 127 - (E + [M > Mc]) and the ratio is at or below the zero cut
// RD(sqrt 2) 2^-(E_max+1) exactly when E + [M > Mc] <= 127 - (E_max + 1).
// Adding 2^23 - 1 - Mc to the bits carries into the exponent exactly when
// M > Mc, so G = clamp((bits + 2^23 - 1 - Mc - (120 << 23)) >> 23, 0, 7)
// is 0 for zero and 7 - e otherwise (E_max = 6, c <= 1 saturates at e = 0).
// The word holds 7 - G per nibble, with the sign bit where G > 0.
__device__ __forceinline__ uint32_t pot4_word(const float (&c)[8], uint32_t sgn, uint32_t cst) {
  uint32_t w = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int t = (int)(__float_as_uint(c[i]) + cst) >> 23;
    const uint32_t gi = (uint32_t)min(max(t, 0), 7);
    w |= gi << (4 * i);
  }
  return (w ^ 0x77777777u) | (sgn & (w + 0x77777777u) & 0x88888888u);
}

// PoT-Mk code word and mantissa-plane bytes of 8 elements from their clamped
// half ratios v_i = min(RN(|x_i| / (2 s)), 1) (0 for NaN): ratios up to 2 on
// the unit interval, so that caller scales with |x| / s in [1, 2) still see
// their mantissa. With v = (1 + M 2^-23) 2^(E-127) and Mc the mantissa of the
// largest cut point (the one between the binade's top value and the next
// binade), F = E + [M > Mc] - 119 (bits + 2^23 - 1 - Mc - (119 << 23), shifted)
// gives the exponent field 7 - clamp(F, 1, 7) for a ratio above the zero cut
// (F >= 8: the top value; F <= 0: the smallest magnitude), 7 for the zero
// code. The mantissa is the number of cut points below m = 1 + M 2^-23 modulo
// 2^k: with t = floor(m 2^k) = 2^k + j0, m lies above the cut between grid
// points j0 and j0 + 1, RD(sqrt(t (t + 1)) / 2^k), exactly when (m 2^k)^2 >
// t (t + 1) (the root is irrational), which one fused multiply-add decides
// by its sign. Saturated ratios take j = 2^k - 1, the smallest magnitude and
// the zero code j = 0. Returns the code word (signs as in pot4_word) and
// writes the K plane bytes (bit i of plane b: bit b of element i's j).
template <int K>
__device__ __forceinline__ uint32_t potmk_word(const float (&v)[8], uint32_t sgn, uint32_t cmk,
                                               uint32_t zc_half, uint32_t (&planes)[K]) {
  constexpr uint32_t n = 1u << K;
  uint32_t w = 0, jw = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t vb = __float_as_uint(v[i]);
    const int f1 = (int)(vb + cmk) >> 23;
    const uint32_t g = (vb > zc_half) ? (uint32_t)min(max(f1, 1), 7) : 0u;
    w |= g << (4 * i);
    const float mn = __uint_as_float((vb & 0x007FFFFFu) | ((127u + K) << 23));  // m 2^k
    const uint32_t j0 = (vb >> (23 - K)) & (n - 1);
    const float t = truncf(mn);                  // 2^k + j0
    const float p = __builtin_fmaf(t, t, t);     // t (t + 1) <= 992, exact
    const uint32_t above = (__builtin_fmaf(mn, mn, -p) > 0.0f) ? 1u : 0u;
    uint32_t j = (j0 + above) & (n - 1);
    j = (f1 > 7) ? n - 1 : j;
    j = (f1 < 1) ? 0u : j;  // also every zero code
    jw |= j << (4 * i);
  }
#pragma unroll
  for (int b = 0; b < K; ++b) {  // bits 4i + b of jw to bit i
    uint32_t x = (jw >> b) & 0x11111111u;
    x = (x | (x >> 3)) & 0x03030303u;
    x = (x | (x >> 6)) & 0x000F000Fu;
    planes[b] = (x | (x >> 12)) & 0xFFu;
  }
  return (w ^ 0x77777777u) | (sgn & (w + 0x77777777u) & 0x88888888u);
}

template <int K, bool HAD>
__global__ __launch_bounds__(kBlock) void encode_pot_kernel(
    const __half* __restrict__ k, int64_t n_rows, int64_t out_stride, int scale_mode,
    float* __restrict__ key_scale, uint8_t* __restrict__ codes_se,
    uint8_t* __restrict__ codes_m, EncodeTables tab) {
  const int lane = threadIdx.x & 63, g = lane & 7, rl = lane >> 3;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t groups = (uint32_t)((n_rows + 7) / 8);
  const uint32_t stride = gridDim.x * (kBlock / 64);
  // K = 0: bits-to-G offset of pot4_word (Mc from the fp32 cut point); K > 0:
  // the offset of potmk_word (the largest cut point) and half the zero cut
  const uint32_t cst =
      K == 0 ? 0x007FFFFFu - (__float_as_uint(tab.cut[0]) & 0x007FFFFFu) - (120u << 23)
             : 0x007FFFFFu - (__float_as_uint(tab.cut[(1 << K) - 1]) & 0x007FFFFFu) - (119u << 23);
  const uint32_t zc_half = __float_as_uint(tab.zero_cut) - (1u << 23);
  // lane parts of the addresses; a group's bases are uniform
  const uint32_t in_off = (uint32_t)(rl * kDim * 2 + 16 * g);
  const int64_t out_row = (int64_t)rl * out_stride;
  const int64_t se_off = out_row * (kDim / 2) + 4 * g;
  for (uint32_t grp_iv = blockIdx.x * (kBlock / 64) + wave; grp_iv < groups;
       grp_iv += stride) {
    // the group index as an opaque uniform value: addresses are rebuilt from
    // it each trip as scalar bases plus the fixed lane offsets
    const uint32_t grp = __builtin_amdgcn_readfirstlane(grp_iv);
    const int64_t row0 = (int64_t)grp * 8;
    const bool valid = row0 + rl < n_rows;  // uniform over the row's 8 lanes
    const char* src = reinterpret_cast<const char*>(k) + row0 * kDim * 2;
    uint4 raw = make_uint4(0u, 0u, 0u, 0u);
    if (valid) raw = *reinterpret_cast<const uint4*>(src + in_off);
    const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
    float x[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __half2float(__ushort_as_half((unsigned short)(w4[i] & 0xFFFFu)));
      x[2 * i + 1] = __half2float(__ushort_as_half((unsigned short)(w4[i] >> 16)));
    }
    if constexpr (HAD) {
      // element 8g + i: butterflies over bits 0..2 of i in registers, over
      // bits 0..2 of g across lanes; fp16 inputs keep every sum exact
      double v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = (double)x[i];
#pragma unroll
      for (int h = 1; h < 8; h <<= 1)
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if ((i & h) == 0) {
            const double p = v[i], q = v[i + h];
            v[i] = p + q;
            v[i + h] = p - q;
          }
#pragma unroll
      for (int hl = 1; hl < 8; hl <<= 1)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const double o = __shfl_xor(v[i], hl, 64);
          v[i] = (g & hl) ? (o - v[i]) : (v[i] + o);
        }
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = (float)(v[i] * 0.125);
    }
    const int64_t orow = (row0 * out_stride) + out_row;
    float s;
    if (scale_mode == 0) {
      // max |x| ignoring NaN (0 for a row of zeros and NaNs)
      s = 0.0f;
#pragma unroll
      for (int i = 0; i < 8; ++i) s = fmaxf(s, fabsf(x[i]));
      s = max_over_8_lanes(s);
    } else {
      s = valid ? key_scale[orow] : 0.0f;
    }
    // The clamped ratio c = min(RN(|x| / ss), 1) per element (ss = s for
    // PoT-4, 2 s for PoT-Mk), NaN -> 0 (zero code), from one correctly
    // rounded reciprocal per row; other scales (zero, negative, NaN,
    // infinite, or too small or too large for a normal reciprocal) divide
    // instead. The quotient q = RN(|x| r) is clamped too: min(q, 1) is still
    // within an ulp of a quotient below 1, any q >= 1 gives c >= 1, and an
    // infinite or NaN q (infinite or NaN x) cannot poison the residual.
    const float ss = K == 0 ? s : 2.0f * s;
    const bool fast = recip_in_range(ss);
    const float r = recip_rn(ss);
    float c[8];
    if (fast) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float a = fabsf(x[i]);
        const float q = clamp01(a * r);
        c[i] = clamp01(__builtin_fmaf(__builtin_fmaf(-q, ss, a), r, q));
      }
    } else {
      // (|x| / 2) / s rounds as |x| / (2 s) and stays finite-safe for huge s
#pragma unroll
      for (int i = 0; i < 8; ++i)
        c[i] = (s > 0.0f) ? clamp01((K == 0 ? fabsf(x[i]) : fabsf(x[i]) * 0.5f) / s) : 0.0f;
    }
    uint32_t sa, sb;  // sign bytes 0x00 / 0xFF of elements 0..3 and 4..7
    if constexpr (HAD) {
      const uint32_t xb[8] = {__float_as_uint(x[0]), __float_as_uint(x[1]),
                              __float_as_uint(x[2]), __float_as_uint(x[3]),
                              __float_as_uint(x[4]), __float_as_uint(x[5]),
                              __float_as_uint(x[6]), __float_as_uint(x[7])};
      // selector 9 / 11: bit 31 of the low / high source, 12: zero byte
      sa = __builtin_amdgcn_perm(xb[1], xb[0], 0x0C0C0B09u) |
           __builtin_amdgcn_perm(xb[3], xb[2], 0x0B090C0Cu);
      sb = __builtin_amdgcn_perm(xb[5], xb[4], 0x0C0C0B09u) |
           __builtin_amdgcn_perm(xb[7], xb[6], 0x0B090C0Cu);
    } else {
      // selectors 8..11: bits 15, 31 of the low and of the high source,
      // the sign bits of the four halves
      sa = __builtin_amdgcn_perm(w4[1], w4[0], 0x0B0A0908u);
      sb = __builtin_amdgcn_perm(w4[3], w4[2], 0x0B0A0908u);
    }
    uint32_t word;
    uint32_t plane[K > 0 ? K : 1];
    if constexpr (K == 0) {
      word = pot4_word(c, sign_nibbles(sa, sb), cst);
    } else {
      word = potmk_word<K>(c, sign_nibbles(sa, sb), cst, zc_half, plane);
    }
    if (valid) {
      const int64_t urow = row0 * out_stride;  // uniform part of orow
      *reinterpret_cast<uint32_t*>(codes_se + urow * (kDim / 2) + se_off) = word;
#pragma unroll
      for (int b = 0; b < K; ++b) codes_m[orow * 8 * K + 8 * b + g] = (uint8_t)plane[b];
      if (scale_mode == 0 && g == 0) key_scale[orow] = s;
    }
  }
}

__global__ __launch_bounds__(kBlock) void encode_int8_kernel(
    const __half* __restrict__ k, int64_t n_rows, int64_t out_stride, int hadamard,
    float* __restrict__ key_scale, int8_t* __restrict__ codes) {
  const int lane = lane_id();
  const int64_t stride = (int64_t)gridDim.x * (kBlock / 64);
  for (int64_t row = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6); row < n_rows;
       row += stride) {  // uniform per wave
    float x = __half2float(k[row * kDim + lane]);
    if (hadamard) x = (float)(wave_fwht64((double)x) * 0.125);
    float step;
    const int c = wave_quantize_int8(x, &step);
    const int64_t orow = row * out_stride;
    codes[orow * kDim + lane] = (int8_t)c;
    if (lane == 0) key_scale[orow] = step;
  }
}

// Value-cache store: token t of sequence s, dim d lives at
// ((s * t_cap + (t/8)*8) * 64 + d * 8 + t % 8) halves. One thread per
// (sequence, 8-token group, dim) gathers the group's 8 tokens of its dim and
// writes them as one 16-byte word (or only the tokens inside [t0, t0+n_tok)
// at the ends of the range). i indexes (sequence, group, dim).
__device__ __forceinline__ void store_value_group(const uint16_t* __restrict__ src, int64_t n_tok,
                                                  int64_t t_cap, int64_t t0, int64_t g_first,
                                                  int64_t n_groups, uint16_t* __restrict__ dst,
                                                  int64_t i) {
  const int d = (int)(i % kDim);
  const int64_t sg = i / kDim;
  const int64_t s = sg / n_groups, g = g_first + sg % n_groups;
  uint16_t* out = dst + (s * t_cap + g * 8) * kDim + d * 8;
  uint16_t vals[8];
  bool full = true;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int64_t t = g * 8 + k;
    const bool in = t >= t0 && t < t0 + n_tok;
    full = full && in;
    vals[k] = in ? src[(s * n_tok + (t - t0)) * kDim + d] : (uint16_t)0;
  }
  if (full) {
    uint4 w;
    w.x = vals[0] | ((uint32_t)vals[1] << 16);
    w.y = vals[2] | ((uint32_t)vals[3] << 16);
    w.z = vals[4] | ((uint32_t)vals[5] << 16);
    w.w = vals[6] | ((uint32_t)vals[7] << 16);
    *reinterpret_cast<uint4*>(out) = w;
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int64_t t = g * 8 + k;
      if (t >= t0 && t < t0 + n_tok) out[k] = vals[k];
    }
  }
}

__global__ __launch_bounds__(256) void store_values_kernel(
    const uint16_t* __restrict__ src, int64_t n_seq, int64_t n_tok, int64_t t_cap, int64_t t0,
    int64_t g_first, int64_t n_groups, uint16_t* __restrict__ dst) {
  const int64_t n = n_seq * n_groups * kDim;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    store_value_group(src, n_tok, t_cap, t0, g_first, n_groups, dst, i);
}

hipError_t launch_store_values(const uint16_t* src, int64_t n_seq, int64_t n_tok, int64_t t_cap,
                               int64_t t0, uint16_t* dst, hipStream_t stream) {
  if (n_seq == 0 || n_tok == 0) return hipSuccess;
  const int64_t g_first = t0 / 8, g_last = (t0 + n_tok - 1) / 8;
  const int64_t n_groups = g_last - g_first + 1;
  const int64_t n = n_seq * n_groups * kDim;
  const int64_t grid = (n + 255) / 256;
  hipLaunchKernelGGL(store_values_kernel, dim3(bounded_grid(grid)), dim3(256), 0, stream, src,
                     n_seq, n_tok, t_cap, t0, g_first, n_groups, dst);
  return hipGetLastError();
}

// One wave per (sequence, token): INT8 quantisation with a power-of-two
// scale and the byte store (Sec. II-E).
__global__ __launch_bounds__(kBlock) void store_values_i8_kernel(
    const uint16_t* __restrict__ src, int64_t n_seq, int64_t n_tok, int64_t t_cap, int64_t t0,
    uint8_t* __restrict__ v_u8, int8_t* __restrict__ v_exp) {
  const int64_t stride = (int64_t)gridDim.x * (kBlock / 64);
  for (int64_t r = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6); r < n_seq * n_tok;
       r += stride) {  // uniform per wave
    const int64_t s = r / n_tok, t = t0 + r % n_tok;
    store_value_token_i8_wave(src + r * kDim, v_u8 + s * t_cap * kDim, v_exp + s * t_cap, t);
  }
}

hipError_t launch_store_values_i8(const uint16_t* src, int64_t n_seq, int64_t n_tok,
                                  int64_t t_cap, int64_t t0, uint8_t* v_u8, int8_t* v_exp,
                                  hipStream_t stream) {
  if (n_seq == 0 || n_tok == 0) return hipSuccess;
  const int64_t rows = n_seq * n_tok;
  const int64_t grid = (rows + kBlock / 64 - 1) / (kBlock / 64);
  hipLaunchKernelGGL(store_values_i8_kernel, dim3(bounded_grid(grid)), dim3(kBlock), 0, stream,
                     src, n_seq, n_tok, t_cap, t0, v_u8, v_exp);
  return hipGetLastError();
}

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, size_t n_words, uint8_t* tail,
                                 size_t tail_bytes) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_words || i < tail_bytes;
       i += (size_t)gridDim.x * blockDim.x) {
    if (i < n_words) p[i] = 0u;
    if (i < tail_bytes) tail[i] = 0;
  }
}

template <int K, bool HAD>
static void launch_encode_pot_t(const uint16_t* k, int64_t n_rows, int64_t out_stride,
                                int scale_mode, float* key_scale, uint8_t* codes_se,
                                uint8_t* codes_m, const EncodeTables& tab, hipStream_t stream) {
  // enough workgroups for several resident waves per SIMD; each wave then
  // loops over row groups, so its set-up is paid once
  const int64_t groups = (n_rows + 7) / 8;
  const int64_t grid =
      std::min<int64_t>((groups + kBlock / 64 - 1) / (kBlock / 64), kEncodeGrid);
  hipLaunchKernelGGL((encode_pot_kernel<K, HAD>), dim3((uint32_t)grid), dim3(kBlock), 0,
                     stream, reinterpret_cast<const __half*>(k), n_rows, out_stride, scale_mode,
                     key_scale, codes_se, codes_m, tab);
}

hipError_t launch_encode_pot(const uint16_t* k, int64_t n_rows, int64_t out_stride,
                             int scale_mode, int hadamard, float* key_scale,
                             uint8_t* codes_se, uint8_t* codes_m, const EncodeTables& tab,
                             hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  auto go = [&](auto k_tag) {
    constexpr int KK = decltype(k_tag)::value;
    if (hadamard)
      launch_encode_pot_t<KK, true>(k, n_rows, out_stride, scale_mode, key_scale, codes_se,
                                    codes_m, tab, stream);
    else
      launch_encode_pot_t<KK, false>(k, n_rows, out_stride, scale_mode, key_scale, codes_se,
                                     codes_m, tab, stream);
  };
  switch (tab.mant_bits) {
    case 0: go(std::integral_constant<int, 0>{}); break;
    case 1: go(std::integral_constant<int, 1>{}); break;
    case 2: go(std::integral_constant<int, 2>{}); break;
    case 3: go(std::integral_constant<int, 3>{}); break;
    case 4: go(std::integral_constant<int, 4>{}); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_encode_int8(const uint16_t* k, int64_t n_rows, int64_t out_stride,
                              int hadamard, float* key_scale, int8_t* codes,
                              hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  const int64_t rows_per_block = kBlock / 64;
  const int64_t grid = (n_rows + rows_per_block - 1) / rows_per_block;
  hipLaunchKernelGGL(encode_int8_kernel, dim3(bounded_grid(grid)), dim3(kBlock), 0, stream,
                     reinterpret_cast<const __half*>(k), n_rows, out_stride, hadamard,
                     key_scale, codes);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  const size_t n_words = bytes / 4;
  const size_t tail = bytes - n_words * 4;
  const size_t n = n_words > tail ? n_words : tail;
  const size_t grid = (n + 255) / 256;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(bounded_grid((int64_t)grid)), dim3(256), 0, stream,
                     reinterpret_cast<uint32_t*>(ptr), n_words,
                     reinterpret_cast<uint8_t*>(ptr) + n_words * 4, tail);
  return hipGetLastError();
}

}  // namespace potattn
