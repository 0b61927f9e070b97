// Key encoders for gfx950: fp16 key rows -> PoT / PoT-Mk codes (Sec. II-A,
// II-D) and -> INT8 uniform codes (the multiply-accumulate comparator).
//
// One wavefront encodes one 64-element key row, one element per lane: a
// 128-byte coalesced fp16 load, an optional exact fp64 Walsh-Hadamard
// butterfly across lanes, a wave max for the per-row scale, a per-lane
// log-nearest decision against fp32 cut points, and packing by lane shuffles
// (sign/exponent nibbles) and ballots (mantissa bit-planes).
#include <hip/hip_fp16.h>

#include <cmath>

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

inline uint32_t bounded_grid(int64_t blocks) {
  return (uint32_t)(blocks < kMaxGrid ? blocks : kMaxGrid);
}

__global__ __launch_bounds__(kBlock) void encode_pot_kernel(
    const __half* __restrict__ k, int64_t n_rows, int64_t out_stride, int scale_mode,
    int hadamard, float* __restrict__ key_scale, uint8_t* __restrict__ codes_se,
    uint8_t* __restrict__ codes_m, EncodeTables tab) {
  const int64_t stride = (int64_t)gridDim.x * (kBlock / 64);
  for (int64_t row = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6); row < n_rows;
       row += stride) {  // uniform per wave
    const int64_t orow = row * out_stride;
    encode_key_row_wave(k + row * kDim, hadamard, scale_mode, key_scale + orow,
                        codes_se + orow * (kDim / 2), codes_m + orow * 8 * tab.mant_bits, tab);
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

hipError_t launch_encode_pot(const uint16_t* k, int64_t n_rows, int64_t out_stride,
                             int scale_mode, int hadamard, float* key_scale,
                             uint8_t* codes_se, uint8_t* codes_m, const EncodeTables& tab,
                             hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  const int64_t rows_per_block = kBlock / 64;
  const int64_t grid = (n_rows + rows_per_block - 1) / rows_per_block;
  hipLaunchKernelGGL(encode_pot_kernel, dim3(bounded_grid(grid)), dim3(kBlock), 0, stream,
                     reinterpret_cast<const __half*>(k), n_rows, out_stride, scale_mode,
                     hadamard, key_scale, codes_se, codes_m, tab);
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
