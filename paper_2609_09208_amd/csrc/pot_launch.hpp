// Host-side launch interface between the C ABI layer (api.cpp) and the
// kernel translation units. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pot_attn.h"

namespace potattn {

constexpr int kMaxHqArg = 128;  // query heads addressable through kernel args

// Encoder tables passed by value as kernel arguments (no device globals).
struct EncodeTables {
  // Cut points between consecutive mantissa grid values inside one binade,
  // scaled to [1, 2): cut[i] = RD_fp32(sqrt((n+i)(n+i+1)) / n), n = 2^k,
  // i = 0..n-1 (the last one separates the binade top from the next binade).
  float cut[16];
  // RD_fp32(2^-(E + 1/2)): ratios at or below it become the exact zero.
  float zero_cut;
  int32_t mant_bits;
};

// Computes EncodeTables for mantissa width k with exact integer square roots.
EncodeTables make_encode_tables(int mant_bits);

hipError_t launch_encode_pot(const uint16_t* k, int64_t n_rows, int64_t out_stride,
                             int scale_mode, int hadamard, float* key_scale,
                             uint8_t* codes_se, uint8_t* codes_m,
                             const EncodeTables& tab, hipStream_t stream);

hipError_t launch_encode_int8(const uint16_t* k, int64_t n_rows, int64_t out_stride,
                              int hadamard, float* key_scale, int8_t* codes,
                              hipStream_t stream);

hipError_t launch_store_values(const uint16_t* src, int64_t n_seq, int64_t n_tok, int64_t t_cap,
                               int64_t t0, uint16_t* dst, hipStream_t stream);

// INT8 values with a power-of-two per-token scale: v_u8 holds v^ + 128
// token-interleaved like the fp16 cache, v_exp one g per cache row.
hipError_t launch_store_values_i8(const uint16_t* src, int64_t n_seq, int64_t n_tok,
                                  int64_t t_cap, int64_t t0, uint8_t* v_u8, int8_t* v_exp,
                                  hipStream_t stream);

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t stream);

// Records a printf-style detail for pot_last_error() on the calling thread and
// returns st (api.cpp).
pot_status report_error(pot_status st, const char* fmt, ...);

// kScoreDs4a: PoT-4 codes decoded to int8 bytes and scored by v_dot4 (a
// multiply path, kept beside the shift path for measurement)
enum ScoreMode : int { kScorePot = 0, kScoreInt8 = 1, kScoreFp16 = 2, kScoreDs4a = 3 };

// Everything one decode launch needs. Passed by value as the kernel argument.
struct DecodeArgs {
  const float* q;
  const uint8_t* codes_se;   // PoT
  const uint8_t* codes_m;    // PoT-Mk planes
  const int8_t* codes_i8;    // INT8 keys
  const uint16_t* k_f16;     // fp16 keys
  const float* key_scale;
  const uint16_t* v;         // fp16 value cache, or
  const uint8_t* v8;         // INT8 value cache (v^ + 128) with
  const int8_t* v_exp;       // one exponent g per row: value v^ 2^-g
  float* out;
  // workspace
  int32_t* qbuf;             // [B*Hkv*n_splits][qstride]: prepared query operands, one
                             // slot per decode workgroup (written and read by it)
  int32_t qstride;           // 32-bit words per slot in qbuf
  int32_t* part_m;           // [B*Hq*S]
  float* part_l;             // [B*Hq*S]
  float* part_o;             // [B*Hq*S*64]
  // debug taps (nullable)
  int8_t* dbg_qhat;
  float* dbg_delta;
  int32_t* dbg_scores;
  int32_t* dbg_m_final;
  int32_t* dbg_m_split;
  // fused append (PoT only; app_k NULL: none): the new token of every
  // (batch, kv head) sequence is encoded into cache row T - 1 and its values
  // stored there by the decode workgroup whose key range holds that row,
  // before it loads any key
  const uint16_t* app_k;     // fp16 [B*Hkv][64]
  const uint16_t* app_v;     // fp16 [B*Hkv][64]
  uint8_t* app_codes_se;     // the cache arrays, written at row T - 1 only
  uint8_t* app_codes_m;
  float* app_key_scale;
  uint16_t* app_v_cache;     // fp16 value cache, or
  uint8_t* app_v8;           // INT8 value cache and
  int8_t* app_v_exp;         // its exponents
  EncodeTables app_tab;
  int64_t t_cap;
  int32_t B, Hq, Hkv, T;
  int32_t n_splits, split_len;
  int32_t frac_bits, hadamard;
  int32_t wg_waves;            // waves per decode workgroup: 4, or pool_waves(...)
  int32_t q_of_kv[kMaxHqArg];  // [Hkv][G] query heads served by each kv head
};

// Waves per workgroup of a decode kernel's CU-wide variant, 0 if it has
// none: four SIMDs times the waves per SIMD that the kernel's registers
// allow (512 per lane and SIMD): the shift-accumulate kernels 4 at k <= 2
// and 3 at k = 3, 4 (fp16 or INT8 values); the decoded-code engines 4, or 3
// for PoT-4 bytes over fp16 values or with power-of-two weights; the INT8
// comparator 3. The fp16 comparator has none: at its two waves per SIMD a
// CU-wide workgroup of 8 waves measured slower than two four-wave ones
// (B = 64, T = 32768: 339.6 against 318.4 us per call).
constexpr int pool_waves(int mode, int mant_bits, int vf) {
  return mode == kScorePot    ? (mant_bits <= 2 ? 16 : 12)
         : mode == kScoreDs4a ? ((mant_bits > 0 || vf == 1) ? 16 : 12)
         : mode == kScoreInt8 ? 12
                              : 0;
}

// Longest key range of one decode call: the decode kernel reads each
// sequence's cache rows through buffer resources with 32-bit byte ranges
// (fp16 values: 128 bytes per key, rounded up to whole 8-key groups).
constexpr int kMaxKeys = (1 << 24) - 8;

// 32-bit words of prepared query operands per kv head for group size G:
// room for the largest layout (32 words per head: 16-bit operand pairs for
// the PoT codes, fp16 pairs for the fp16 comparator) plus the G per-head
// score factors.
constexpr int query_words(int G) { return (33 * G + 63) / 64 * 64; }

// Resident workgroups per CU of the (non-debug) decode kernel for this
// variant (pool: its CU-wide variant), from the HIP occupancy calculator; 0 if
// the query fails.
int decode_occupancy(int mode, int G, int mant_bits, int vf, bool pool);

// vf: value format. 0: fp16 value cache (a.v); 1: INT8 value cache (a.v8,
// a.v_exp); 2: INT8 values with the power-of-two weights of eq. logsm.
// Formats 1 and 2 exist for the score modes kScorePot and kScoreDs4a only.
// ev_begin / ev_end (may be null) are recorded on the stream right before and
// right after the decode kernel.
hipError_t launch_decode(int mode, int G, int mant_bits, bool debug, int vf,
                         const DecodeArgs& a, hipStream_t stream, hipEvent_t ev_begin = nullptr,
                         hipEvent_t ev_end = nullptr);

// The launch and occupancy query of one score mode and value format; each
// mode's kernels are instantiated in a translation unit of their own.
template <int MODE, int VF>
hipError_t launch_mode_vf(int G, int mant_bits, bool debug, const DecodeArgs& a,
                          hipStream_t stream, hipEvent_t e0, hipEvent_t e1);
template <int MODE, int VF>
int occupancy_mode_vf(int G, int mant_bits, bool pool);

}  // namespace potattn
