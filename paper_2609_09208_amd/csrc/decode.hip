// Split-K decode attention for gfx950 over a PoT / INT8 / fp16 key cache.
//
// Grid (n_splits, Hkv, B), 256 threads (4 wave64). A workgroup owns one key
// range of one (batch, kv-head) sequence and all G query heads that share the
// kv head (GQA), so every code byte and value byte is read from HBM once per
// workgroup and reused G times.
//
// Per tile of 256 keys:
//  1. score: thread t owns key t. PoT (Sec. II-B eq. sac): the row's 32 code
//     bytes arrive as two 16-byte loads; per element the exponent gives the
//     funnel-shift amount sh = e + 25, so v_alignbit(q, 0, sh) = q << (7 - e)
//     for e <= 6 and 0 for the zero code e = 7 (sh = 32 = 0 mod 32). The sign
//     is applied as (t ^ s) + acc (v_xad_u32) with s in {0, -1}, and the
//     missing +1 per negative element is added once per key from a popcount
//     of the sign bits. Mantissa bit b of PoT-Mk adds alignbit(q << b, 0,
//     sh & -bit). Every shift is a left shift (eq. exact) and the int32 sum is
//     exact; it is taken at internal head-room 7 and rescaled exactly to F.
//  2. log2 domain: x = fl32(fl32(float(acc) * s) * c), c = fl32(fl32(Delta *
//     log2 e) * 2^-(F+k+3)), in this fixed fp32 order.
//  3. integer running maximum M = max(M, ceil(max x)) per head (eq. logsm);
//     a rise rescales the running sums by the exact power of two 2^(M_old -
//     M_new).
//  4. A.V: weights p = 2^(x - M) staged in LDS; thread (key group, 8 dims)
//     streams 16-byte fp16 value loads and accumulates G x 8 fp32 sums.
// After its range, a workgroup writes (M_s, l_s, o_s) per head; the last
// workgroup of a (batch, kv-head) to finish (split-completion counter) merges
// the splits with exact 2^(M_s - M) weights and resets the counter.
#include <hip/hip_fp16.h>

#include <climits>

#include "pot_device.hpp"
#include "pot_launch.hpp"

namespace potattn {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

template <int MODE, int K>
struct QLayout {
  // 32-bit query words per element-group and head held in LDS.
  static constexpr int kWords = MODE == kScorePot ? (K + 1) * kDim
                                : MODE == kScoreInt8 ? kDim / 4
                                                     : kDim / 2;
};

template <int MODE, int G, int K, bool DEBUG>
__global__ __launch_bounds__(kBlock) void decode_kernel(const DecodeArgs a) {
  constexpr int NQW = QLayout<MODE, K>::kWords;
  __shared__ int32_t s_q[NQW][G];
  __shared__ float s_c[G];
  __shared__ float s_x[kTile][G];
  __shared__ float s_red[4][G];
  __shared__ float s_o[4][G][kDim];
  __shared__ float s_l[4][G];
  __shared__ int s_m[G];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int64_t row0 = ((int64_t)b * a.Hkv + kvh) * a.t_cap;

  // ---- prologue: rotate and quantise this kv head's G query vectors ------
  for (int h = wave; h < G; h += 4) {
    const int64_t bq = (int64_t)b * a.Hq + a.q_of_kv[kvh * G + h];
    float qv = a.q[bq * kDim + lane];
    if constexpr (MODE == kScoreFp16) {
      const uint32_t bits = __half_as_ushort(__float2half_rn(qv));
      const uint32_t other = __shfl_xor(bits, 1, 64);
      if ((lane & 1) == 0) s_q[lane >> 1][h] = (int32_t)(bits | (other << 16));
      if (lane == 0) s_c[h] = __fmul_rn(log2e_f32(), 0.125f);
    } else {
      if (a.hadamard) qv = (float)(wave_fwht64((double)qv) * 0.125);
      float step;
      const int qi = wave_quantize_int8(qv, &step);
      if constexpr (MODE == kScorePot) {
#pragma unroll
        for (int bb = 0; bb <= K; ++bb) s_q[bb * kDim + lane][h] = qi * (1 << bb);
        if (lane == 0)
          s_c[h] = __fmul_rn(__fmul_rn(step, log2e_f32()),
                             __builtin_amdgcn_ldexpf(1.0f, -(a.frac_bits + K + 3)));
      } else {
        uint32_t word = (uint32_t)(qi & 0xFF) << (8 * (lane & 3));
        word |= __shfl_xor(word, 1, 64);
        word |= __shfl_xor(word, 2, 64);
        if ((lane & 3) == 0) s_q[lane >> 2][h] = (int32_t)word;
        if (lane == 0) s_c[h] = __fmul_rn(__fmul_rn(step, log2e_f32()), 0.125f);
      }
      if constexpr (DEBUG) {
        if (split == 0) {
          if (a.dbg_qhat) a.dbg_qhat[bq * kDim + lane] = (int8_t)qi;
          if (a.dbg_delta && lane == 0) a.dbg_delta[bq] = step;
        }
      }
    }
  }
  __syncthreads();

  const int t_begin = split * a.split_len;
  const int t_end = min(a.T, t_begin + a.split_len);
  const int kg = tid >> 3, d8 = tid & 7;

  int m_run[G];
  float l_acc[G], o_acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_run[h] = INT_MIN;
    l_acc[h] = 0.0f;
#pragma unroll
    for (int dd = 0; dd < 8; ++dd) o_acc[h][dd] = 0.0f;
  }

  for (int tile = t_begin; tile < t_end; tile += kTile) {
    const int t = tile + tid;
    float xs[G];
    if (t < t_end) {
      const int64_t row = row0 + t;
      if constexpr (MODE == kScorePot) {
        const uint4* cp = reinterpret_cast<const uint4*>(a.codes_se + row * (kDim / 2));
        const uint4 c0 = cp[0], c1 = cp[1];
        const uint32_t w[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
        uint64_t pl[K > 0 ? K : 1];
#pragma unroll
        for (int bb = 0; bb < K; ++bb)
          pl[bb] = reinterpret_cast<const uint64_t*>(a.codes_m + row * 8 * K)[bb];
        int nneg = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) nneg += __popc(w[i] & 0x88888888u);
        uint32_t acc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = 0u;
#pragma unroll
        for (int m = 0; m < kDim; ++m) {
          const uint32_t word = w[m >> 3];
          const int pos = 4 * (m & 7);
          const uint32_t sh = ((word >> pos) & 7u) + 25u;
          const uint32_t sgn = (uint32_t)((int32_t)(word << (28 - pos)) >> 31);
          uint32_t shb[K > 0 ? K : 1];
#pragma unroll
          for (int bb = 0; bb < K; ++bb)
            shb[bb] = sh & (uint32_t)(-(int32_t)((pl[bb] >> m) & 1u));
#pragma unroll
          for (int h = 0; h < G; ++h) {
            uint32_t term = __builtin_amdgcn_alignbit((uint32_t)s_q[K * kDim + m][h], 0u, sh);
#pragma unroll
            for (int bb = 0; bb < K; ++bb)
              term += __builtin_amdgcn_alignbit((uint32_t)s_q[bb * kDim + m][h], 0u, shb[bb]);
            acc[h] = (term ^ sgn) + acc[h];
          }
        }
        const float s = a.key_scale[row];
#pragma unroll
        for (int h = 0; h < G; ++h) {
          int32_t v = (int32_t)(acc[h] + (uint32_t)nneg);
          v = a.frac_bits >= kFInt ? (int32_t)((uint32_t)v << (a.frac_bits - kFInt))
                                   : (v >> (kFInt - a.frac_bits));
          xs[h] = __fmul_rn(__fmul_rn((float)v, s), s_c[h]);
          if constexpr (DEBUG) {
            if (a.dbg_scores)
              a.dbg_scores[((int64_t)b * a.Hq + a.q_of_kv[kvh * G + h]) * a.T + t] = v;
          }
        }
      } else if constexpr (MODE == kScoreInt8) {
        const int4* kp = reinterpret_cast<const int4*>(a.codes_i8 + row * kDim);
        int32_t kw[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int4 v4 = kp[i];
          kw[4 * i] = v4.x;
          kw[4 * i + 1] = v4.y;
          kw[4 * i + 2] = v4.z;
          kw[4 * i + 3] = v4.w;
        }
        int32_t acc[G];
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h] = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i)
#pragma unroll
          for (int h = 0; h < G; ++h) acc[h] = __builtin_amdgcn_sdot4(s_q[i][h], kw[i], acc[h], false);
        const float s = a.key_scale[row];
#pragma unroll
        for (int h = 0; h < G; ++h) {
          xs[h] = __fmul_rn(__fmul_rn((float)acc[h], s), s_c[h]);
          if constexpr (DEBUG) {
            if (a.dbg_scores)
              a.dbg_scores[((int64_t)b * a.Hq + a.q_of_kv[kvh * G + h]) * a.T + t] = acc[h];
          }
        }
      } else {
        const uint4* kp = reinterpret_cast<const uint4*>(a.k_f16 + row * kDim);
        uint32_t kw[32];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint4 v4 = kp[i];
          kw[4 * i] = v4.x;
          kw[4 * i + 1] = v4.y;
          kw[4 * i + 2] = v4.z;
          kw[4 * i + 3] = v4.w;
        }
        float dot[G];
#pragma unroll
        for (int h = 0; h < G; ++h) dot[h] = 0.0f;
#pragma unroll
        for (int i = 0; i < 32; ++i)
#pragma unroll
          for (int h = 0; h < G; ++h)
            dot[h] = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, s_q[i][h]),
                                            __builtin_bit_cast(half2v, kw[i]), dot[h], false);
#pragma unroll
        for (int h = 0; h < G; ++h) xs[h] = __fmul_rn(dot[h], s_c[h]);
      }
    } else {
#pragma unroll
      for (int h = 0; h < G; ++h) xs[h] = -INFINITY;
    }

    // tile maximum per head
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mx = wave_max(xs[h]);
      if (lane == 0) s_red[wave][h] = mx;
    }
    __syncthreads();
    float scale[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mt = fmaxf(fmaxf(s_red[0][h], s_red[1][h]), fmaxf(s_red[2][h], s_red[3][h]));
      const int m_new = max(m_run[h], (int)ceilf(mt));
      scale[h] = m_run[h] == INT_MIN ? 0.0f : __builtin_amdgcn_ldexpf(1.0f, m_run[h] - m_new);
      m_run[h] = m_new;
    }
    // weights of this thread's own key
#pragma unroll
    for (int h = 0; h < G; ++h)
      s_x[tid][h] = (t < t_end) ? __builtin_amdgcn_exp2f(xs[h] - (float)m_run[h]) : 0.0f;
    __syncthreads();

    // A.V: thread (kg, d8) takes keys kg, kg+32, ... and dims 8*d8 .. 8*d8+7
#pragma unroll
    for (int h = 0; h < G; ++h) {
      l_acc[h] *= scale[h];
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) o_acc[h][dd] *= scale[h];
    }
#pragma unroll 2
    for (int i = 0; i < kTile / 32; ++i) {
      const int tl = kg + 32 * i;
      if (tile + tl < t_end) {
        const uint4 vv = *reinterpret_cast<const uint4*>(a.v + (row0 + tile + tl) * kDim + 8 * d8);
        const uint32_t vw[4] = {vv.x, vv.y, vv.z, vv.w};
        float vf[8];
#pragma unroll
        for (int i2 = 0; i2 < 4; ++i2) {
          const half2v hv = __builtin_bit_cast(half2v, vw[i2]);
          vf[2 * i2] = (float)hv.x;
          vf[2 * i2 + 1] = (float)hv.y;
        }
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float p = s_x[tl][h];
          l_acc[h] += p;
#pragma unroll
          for (int dd = 0; dd < 8; ++dd) o_acc[h][dd] = fmaf(p, vf[dd], o_acc[h][dd]);
        }
      }
    }
    __syncthreads();
  }

  // ---- reduce this workgroup's partial sums over key groups --------------
#pragma unroll
  for (int h = 0; h < G; ++h) {
#pragma unroll
    for (int dd = 0; dd < 8; ++dd) {
      float v = o_acc[h][dd];
      v += __shfl_xor(v, 8, 64);
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      if (lane < 8) s_o[wave][h][8 * lane + dd] = v;
    }
    float l = l_acc[h];
    l += __shfl_xor(l, 8, 64);
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (lane == 0) s_l[wave][h] = l;
  }
  if (tid == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) s_m[h] = m_run[h];
  }
  __syncthreads();

  const int S = a.n_splits;
  for (int idx = tid; idx < G * kDim; idx += kBlock) {
    const int h = idx / kDim, d = idx % kDim;
    const int64_t bq = (int64_t)b * a.Hq + a.q_of_kv[kvh * G + h];
    const float o = (s_o[0][h][d] + s_o[1][h][d]) + (s_o[2][h][d] + s_o[3][h][d]);
    const float l = (s_l[0][h] + s_l[1][h]) + (s_l[2][h] + s_l[3][h]);
    if (S == 1) {
      a.out[bq * kDim + d] = o / l;
      if constexpr (DEBUG) {
        if (d == 0 && a.dbg_m_final) a.dbg_m_final[bq] = s_m[h];
        if (d == 0 && a.dbg_m_split) a.dbg_m_split[bq] = s_m[h];
      }
    } else {
      const int64_t ps = bq * S + split;
      a.part_o[ps * kDim + d] = o;
      if (d == 0) {
        a.part_l[ps] = l;
        a.part_m[ps] = s_m[h];
        if constexpr (DEBUG) {
          if (a.dbg_m_split) a.dbg_m_split[ps] = s_m[h];
        }
      }
    }
  }
  if (S == 1) return;

  // ---- split combine by the last workgroup of this (batch, kv head) -------
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = atomicAdd(&a.counters[(int64_t)b * a.Hkv + kvh], 1u);
    s_last = (old == (uint32_t)(S - 1));
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  for (int idx = tid; idx < G * kDim; idx += kBlock) {
    const int h = idx / kDim, d = idx % kDim;
    const int64_t bq = (int64_t)b * a.Hq + a.q_of_kv[kvh * G + h];
    int M = INT_MIN;
    for (int s = 0; s < S; ++s) M = max(M, a.part_m[bq * S + s]);
    float L = 0.0f, O = 0.0f;
    for (int s = 0; s < S; ++s) {
      const float f = __builtin_amdgcn_ldexpf(1.0f, a.part_m[bq * S + s] - M);
      L = fmaf(f, a.part_l[bq * S + s], L);
      O = fmaf(f, a.part_o[(bq * S + s) * kDim + d], O);
    }
    a.out[bq * kDim + d] = O / L;
    if constexpr (DEBUG) {
      if (d == 0 && a.dbg_m_final) a.dbg_m_final[bq] = M;
    }
  }
  if (tid == 0) a.counters[(int64_t)b * a.Hkv + kvh] = 0u;
}

template <int MODE, int G, int K, bool DEBUG>
static hipError_t launch_t(const DecodeArgs& a, hipStream_t stream) {
  const dim3 grid((uint32_t)a.n_splits, (uint32_t)a.Hkv, (uint32_t)a.B);
  hipLaunchKernelGGL((decode_kernel<MODE, G, K, DEBUG>), grid, dim3(kBlock), 0, stream, a);
  return hipGetLastError();
}

template <int MODE, int G, bool DEBUG>
static hipError_t launch_k(int mant_bits, const DecodeArgs& a, hipStream_t stream) {
  if constexpr (MODE != kScorePot) {
    return launch_t<MODE, G, 0, DEBUG>(a, stream);
  } else {
    switch (mant_bits) {
      case 0: return launch_t<MODE, G, 0, DEBUG>(a, stream);
      case 1: return launch_t<MODE, G, 1, DEBUG>(a, stream);
      case 2: return launch_t<MODE, G, 2, DEBUG>(a, stream);
      case 3: return launch_t<MODE, G, 3, DEBUG>(a, stream);
      case 4: return launch_t<MODE, G, 4, DEBUG>(a, stream);
      default: return hipErrorInvalidValue;
    }
  }
}

template <int MODE, bool DEBUG>
static hipError_t launch_g(int G, int mant_bits, const DecodeArgs& a, hipStream_t stream) {
  switch (G) {
    case 1: return launch_k<MODE, 1, DEBUG>(mant_bits, a, stream);
    case 2: return launch_k<MODE, 2, DEBUG>(mant_bits, a, stream);
    case 4: return launch_k<MODE, 4, DEBUG>(mant_bits, a, stream);
    case 8: return launch_k<MODE, 8, DEBUG>(mant_bits, a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_decode(int mode, int G, int mant_bits, bool debug, const DecodeArgs& a,
                         hipStream_t stream) {
  switch (mode) {
    case kScorePot:
      return debug ? launch_g<kScorePot, true>(G, mant_bits, a, stream)
                   : launch_g<kScorePot, false>(G, mant_bits, a, stream);
    case kScoreInt8:
      return debug ? launch_g<kScoreInt8, true>(G, 0, a, stream)
                   : launch_g<kScoreInt8, false>(G, 0, a, stream);
    case kScoreFp16:
      return launch_g<kScoreFp16, false>(G, 0, a, stream);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace potattn
