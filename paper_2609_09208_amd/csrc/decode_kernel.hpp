// Split-K decode attention for gfx950 over a PoT / INT8 / fp16 key cache.
//
// Grid (n_splits, Hkv, B), 256 threads = 4 wave64, or in the CU-wide variant
// one workgroup of pool_waves(...) waves per CU. A workgroup owns one key
// range of one (batch, kv-head) sequence and all G query heads sharing that
// kv head (GQA), so every code and value byte is read from HBM once and used
// G times. Inside the workgroup each wave streams its own 64-key tiles
// (tile j of the range goes to wave j % 4; in the CU-wide variant the waves
// claim tiles from a counter in LDS) with the next tile's codes (and, for
// the short score cores, value fragments) prefetched into registers while
// the current one is processed; waves only meet at the end to merge their
// partial sums.
//
// Per 64-key tile and wave:
//  1. Scores, one key per lane (Sec. II-B eq. sac). PoT-4: the key's 32 code
//     bytes arrive as two 16-byte loads. Each query operand holds two
//     elements of one head as signed 16-bit halves, q 2^7 (prepared once per
//     kv head, read through the scalar cache in chunks of two element pairs,
//     each requested while the previous one is used). v_pk_ashrrev_i16
//     (inline assembly, which reads the exponent nibbles in place) shifts
//     each half by its element's exponent e:
//     q 2^7 >> e = q 2^(7 - e), exact since the low 7 bits are clear, so
//     every product q 2^(7 - e) is formed by the shifter with head-room
//     F_int = 7 >= e (eq. exact). v_dot2_i32_i16 then applies the signs and
//     sums both halves into the int32 score: it is the dot unit's integer
//     multiply-add, used here with weights sigma in {-1, +1} (0 for the zero
//     code), so its multipliers only ever see -1, 0 or +1. PoT-Mk (Sec.
//     II-D) adds one sum per mantissa bit plane b over the same shifted
//     operands, with weight sigma where bit b of the element's mantissa is
//     set and 0 elsewhere; the key's sum is 2^k S_lead + sum_b 2^b S_b, the
//     per-bit shifts of eq. sac regrouped by plane. The decoded-code engines
//     (a multiply path) instead decode each code once per key into dot-unit
//     weights shared by all G heads: PoT-4 into int8 bytes sigma 2^(6 - e)
//     for v_dot4_i32_i8, PoT-Mk into 16-bit sigma (2^k + j) 2^(7 - e) for
//     v_dot2_i32_i16; the int32 sums equal the shift-accumulate ones.
//  2. x = fl32(fl32(float(acc) * s) * c), c = fl32(fl32(Delta * log2 e) *
//     2^-(F+k+3)) in this order; x is staged transposed in wave-private LDS.
//  3. Integer running maximum M = max(M, ceil(max x)) per head (eq. logsm);
//     when it rises the accumulators are rescaled by the exact power of two
//     2^(M_old - M_new).
//  4. A.V on the matrix cores: P (16 rows = 8 heads x {fp16 high part, fp16
//     low part} of p = 2^(x - M + 12)) times V (fp16) with
//     v_mfma_f32_16x16x32_f16, fp32 accumulation; a fifth column block of
//     ones yields the row sums l. The value cache is stored token-interleaved
//     ([t/8][d][t%8]) so a lane's 16-byte load is exactly its B fragment.
// With one split the workgroup writes O directly; otherwise it writes its
// (M_s, l_s, o_s) and a small combine kernel merges the splits with exact
// 2^(M_s - M) weights. (A last-workgroup merge inside this kernel would need
// an agent-scope release/acquire per workgroup, which on a multi-XCD part
// writes back and invalidates the XCD's L2 each time and serialises.)
// (Kernel templates; the instantiations live in decode_pot*.hip,
// decode_dot.hip and decode_cmp.hip, one translation unit per score mode and
// value format.)
#pragma once

#include <hip/hip_fp16.h>

#include <climits>
#include <type_traits>

#include "pot_device.hpp"
#include "pot_launch.hpp"

namespace potattn {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Shift-accumulate of one element pair for G heads (G = 2, 4 or 8): each
// head's uniform word q[h] (operands q 2^7 of elements 8c + n and 8c + n + 4)
// is shifted right arithmetically per half by the low four bits of the
// matching half of sh, and the result is added into the head's int32 sum
// a[h] by v_dot2_i32_i16 with the pair's weights w (1, -1 or 0 per half); the
// first pair of a key starts the sums from 0. v_pk_ashrrev_i16 reads only
// those four bits, so the caller need not clear the bits above them (a C++
// vector shift needs every amount below 16 and so costs a mask). Heads go two
// at a time, both shifts before both sums, so each v_dot2 reads a result
// written two instructions earlier; one block for all G heads leaves the
// compiler no boundary between them at which to add wait states.
#define POT_SAC_SH(t, h) "v_pk_ashrrev_i16 %" #t ", %[sh], %[q" #h "]\n\t"
#define POT_SAC_D0(h, t) "v_dot2_i32_i16 %[a" #h "], %" #t ", %[w], 0\n\t"
#define POT_SAC_DC(h, t) "v_dot2c_i32_i16 %[a" #h "], %" #t ", %[w]\n\t"
#define POT_SAC_2(D, x, y) POT_SAC_SH(0, x) POT_SAC_SH(1, y) D(x, 0) D(y, 1)
template <int G, bool kFirst>
__device__ __forceinline__ void sac_heads(int32_t* a, const uint32_t* q, uint32_t sh, uint32_t w) {
  static_assert(G == 2 || G == 4 || G == 8, "two, four or eight heads");
  uint32_t t0, t1;
  if constexpr (G == 2) {
    if constexpr (kFirst)
      asm(POT_SAC_2(POT_SAC_D0, 0, 1)
          : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[0]), [a1] "=&v"(a[1])
          : [sh] "v"(sh), [w] "v"(w), [q0] "s"(q[0]), [q1] "s"(q[1]));
    else
      asm(POT_SAC_2(POT_SAC_DC, 0, 1)
          : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[0]), [a1] "+v"(a[1])
          : [sh] "v"(sh), [w] "v"(w), [q0] "s"(q[0]), [q1] "s"(q[1]));
  } else if constexpr (G == 4) {
    if constexpr (kFirst)
      asm(POT_SAC_2(POT_SAC_D0, 0, 1) POT_SAC_2(POT_SAC_D0, 2, 3)
          : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[0]), [a1] "=&v"(a[1]), [a2] "=&v"(a[2]),
            [a3] "=&v"(a[3])
          : [sh] "v"(sh), [w] "v"(w), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]),
            [q3] "s"(q[3]));
    else
      asm(POT_SAC_2(POT_SAC_DC, 0, 1) POT_SAC_2(POT_SAC_DC, 2, 3)
          : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[0]), [a1] "+v"(a[1]), [a2] "+v"(a[2]),
            [a3] "+v"(a[3])
          : [sh] "v"(sh), [w] "v"(w), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]),
            [q3] "s"(q[3]));
  } else {
    if constexpr (kFirst)
      asm(POT_SAC_2(POT_SAC_D0, 0, 1) POT_SAC_2(POT_SAC_D0, 2, 3)
              POT_SAC_2(POT_SAC_D0, 4, 5) POT_SAC_2(POT_SAC_D0, 6, 7)
          : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[0]), [a1] "=&v"(a[1]), [a2] "=&v"(a[2]),
            [a3] "=&v"(a[3]), [a4] "=&v"(a[4]), [a5] "=&v"(a[5]), [a6] "=&v"(a[6]),
            [a7] "=&v"(a[7])
          : [sh] "v"(sh), [w] "v"(w), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]),
            [q3] "s"(q[3]), [q4] "s"(q[4]), [q5] "s"(q[5]), [q6] "s"(q[6]), [q7] "s"(q[7]));
    else
      asm(POT_SAC_2(POT_SAC_DC, 0, 1) POT_SAC_2(POT_SAC_DC, 2, 3)
              POT_SAC_2(POT_SAC_DC, 4, 5) POT_SAC_2(POT_SAC_DC, 6, 7)
          : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[0]), [a1] "+v"(a[1]), [a2] "+v"(a[2]),
            [a3] "+v"(a[3]), [a4] "+v"(a[4]), [a5] "+v"(a[5]), [a6] "+v"(a[6]),
            [a7] "+v"(a[7])
          : [sh] "v"(sh), [w] "v"(w), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]),
            [q3] "s"(q[3]), [q4] "s"(q[4]), [q5] "s"(q[5]), [q6] "s"(q[6]), [q7] "s"(q[7]));
  }
}
// The same for one mantissa bit plane (k = 1): each shifted operand also goes
// into the head's plane sum c[h] with the plane weights m (sigma where the
// element's mantissa bit is set, else 0).
#define POT_SAC1_D0(h, t)                                 \
  "v_dot2_i32_i16 %[a" #h "], %" #t ", %[w], 0\n\t" \
  "v_dot2_i32_i16 %[c" #h "], %" #t ", %[m], 0\n\t"
#define POT_SAC1_DC(h, t)                              \
  "v_dot2c_i32_i16 %[a" #h "], %" #t ", %[w]\n\t" \
  "v_dot2c_i32_i16 %[c" #h "], %" #t ", %[m]\n\t"
template <int G, bool kFirst>
__device__ __forceinline__ void sac_heads_m1(int32_t* a, int32_t* c, const uint32_t* q, uint32_t sh,
                                             uint32_t w, uint32_t m) {
  static_assert(G == 2 || G == 4 || G == 8, "two, four or eight heads");
  uint32_t t0, t1;
  if constexpr (G == 2) {
    if constexpr (kFirst)
      asm(POT_SAC_2(POT_SAC1_D0, 0, 1)
          : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[0]), [a1] "=&v"(a[1]), [c0] "=&v"(c[0]), [c1] "=&v"(c[1])
          : [sh] "v"(sh), [w] "v"(w), [m] "v"(m), [q0] "s"(q[0]), [q1] "s"(q[1]));
    else
      asm(POT_SAC_2(POT_SAC1_DC, 0, 1)
          : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[0]), [a1] "+v"(a[1]), [c0] "+v"(c[0]), [c1] "+v"(c[1])
          : [sh] "v"(sh), [w] "v"(w), [m] "v"(m), [q0] "s"(q[0]), [q1] "s"(q[1]));
  } else if constexpr (G == 4) {
    if constexpr (kFirst)
      asm(POT_SAC_2(POT_SAC1_D0, 0, 1) POT_SAC_2(POT_SAC1_D0, 2, 3)
          : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[0]), [a1] "=&v"(a[1]), [a2] "=&v"(a[2]), [a3] "=&v"(a[3]), [c0] "=&v"(c[0]), [c1] "=&v"(c[1]), [c2] "=&v"(c[2]), [c3] "=&v"(c[3])
          : [sh] "v"(sh), [w] "v"(w), [m] "v"(m), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]));
    else
      asm(POT_SAC_2(POT_SAC1_DC, 0, 1) POT_SAC_2(POT_SAC1_DC, 2, 3)
          : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[0]), [a1] "+v"(a[1]), [a2] "+v"(a[2]), [a3] "+v"(a[3]), [c0] "+v"(c[0]), [c1] "+v"(c[1]), [c2] "+v"(c[2]), [c3] "+v"(c[3])
          : [sh] "v"(sh), [w] "v"(w), [m] "v"(m), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]));
  } else if constexpr (G == 8) {
    if constexpr (kFirst)
      asm(POT_SAC_2(POT_SAC1_D0, 0, 1) POT_SAC_2(POT_SAC1_D0, 2, 3) POT_SAC_2(POT_SAC1_D0, 4, 5) POT_SAC_2(POT_SAC1_D0, 6, 7)
          : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[0]), [a1] "=&v"(a[1]), [a2] "=&v"(a[2]), [a3] "=&v"(a[3]), [a4] "=&v"(a[4]), [a5] "=&v"(a[5]), [a6] "=&v"(a[6]), [a7] "=&v"(a[7]), [c0] "=&v"(c[0]), [c1] "=&v"(c[1]), [c2] "=&v"(c[2]), [c3] "=&v"(c[3]), [c4] "=&v"(c[4]), [c5] "=&v"(c[5]), [c6] "=&v"(c[6]), [c7] "=&v"(c[7])
          : [sh] "v"(sh), [w] "v"(w), [m] "v"(m), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]), [q4] "s"(q[4]), [q5] "s"(q[5]), [q6] "s"(q[6]), [q7] "s"(q[7]));
    else
      asm(POT_SAC_2(POT_SAC1_DC, 0, 1) POT_SAC_2(POT_SAC1_DC, 2, 3) POT_SAC_2(POT_SAC1_DC, 4, 5) POT_SAC_2(POT_SAC1_DC, 6, 7)
          : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[0]), [a1] "+v"(a[1]), [a2] "+v"(a[2]), [a3] "+v"(a[3]), [a4] "+v"(a[4]), [a5] "+v"(a[5]), [a6] "+v"(a[6]), [a7] "+v"(a[7]), [c0] "+v"(c[0]), [c1] "+v"(c[1]), [c2] "+v"(c[2]), [c3] "+v"(c[3]), [c4] "+v"(c[4]), [c5] "+v"(c[5]), [c6] "+v"(c[6]), [c7] "+v"(c[7])
          : [sh] "v"(sh), [w] "v"(w), [m] "v"(m), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]), [q4] "s"(q[4]), [q5] "s"(q[5]), [q6] "s"(q[6]), [q7] "s"(q[7]));
  }
}
#undef POT_SAC1_DC
#undef POT_SAC1_D0
// The same for k = 2, 3 or 4 mantissa bit planes, H = 2 or 4 heads per block
// (the operand count of one statement is limited): plane b's sum of head h is
// c[b][h0 + h], with the plane weights m[b].
#define POT_DOT0(acc, t, wt) "v_dot2_i32_i16 %[" acc "], %" #t ", %[" wt "], 0\n\t"
#define POT_DOTC(acc, t, wt) "v_dot2c_i32_i16 %[" acc "], %" #t ", %[" wt "]\n\t"
#define POT_HEAD_K2(D, h, t) D("a" #h, t, "w") D("c0" #h, t, "m0") D("c1" #h, t, "m1")
#define POT_HEAD_K3(D, h, t) POT_HEAD_K2(D, h, t) D("c2" #h, t, "m2")
#define POT_HEAD_K4(D, h, t) POT_HEAD_K3(D, h, t) D("c3" #h, t, "m3")
#define POT_PAIR(HK, D, x, y) POT_SAC_SH(0, x) POT_SAC_SH(1, y) HK(D, x, 0) HK(D, y, 1)
template <int H, int K, int G, bool kFirst>
__device__ __forceinline__ void sac_heads_mk(int32_t* a, int32_t (*c)[G], int h0, const uint32_t* q,
                                             uint32_t sh, uint32_t w, const uint32_t* m) {
  static_assert((H == 2 && K >= 2 && K <= 4) || (H == 4 && (K == 2 || K == 3)),
                "two heads with two to four planes, or four heads with two or three");
  uint32_t t0, t1;
  if constexpr (H == 2 && K == 2 && kFirst) {
    asm(POT_PAIR(POT_HEAD_K2, POT_DOT0, 0, 1)
        : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[h0 + 0]), [a1] "=&v"(a[h0 + 1]),
          [c00] "=&v"(c[0][h0 + 0]), [c01] "=&v"(c[0][h0 + 1]), [c10] "=&v"(c[1][h0 + 0]),
          [c11] "=&v"(c[1][h0 + 1])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [q0] "s"(q[0]),
          [q1] "s"(q[1]));
  } else if constexpr (H == 2 && K == 2 && !kFirst) {
    asm(POT_PAIR(POT_HEAD_K2, POT_DOTC, 0, 1)
        : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[h0 + 0]), [a1] "+v"(a[h0 + 1]),
          [c00] "+v"(c[0][h0 + 0]), [c01] "+v"(c[0][h0 + 1]), [c10] "+v"(c[1][h0 + 0]),
          [c11] "+v"(c[1][h0 + 1])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [q0] "s"(q[0]),
          [q1] "s"(q[1]));
  } else if constexpr (H == 2 && K == 3 && kFirst) {
    asm(POT_PAIR(POT_HEAD_K3, POT_DOT0, 0, 1)
        : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[h0 + 0]), [a1] "=&v"(a[h0 + 1]),
          [c00] "=&v"(c[0][h0 + 0]), [c01] "=&v"(c[0][h0 + 1]), [c10] "=&v"(c[1][h0 + 0]),
          [c11] "=&v"(c[1][h0 + 1]), [c20] "=&v"(c[2][h0 + 0]), [c21] "=&v"(c[2][h0 + 1])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [m2] "v"(m[2]),
          [q0] "s"(q[0]), [q1] "s"(q[1]));
  } else if constexpr (H == 2 && K == 3 && !kFirst) {
    asm(POT_PAIR(POT_HEAD_K3, POT_DOTC, 0, 1)
        : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[h0 + 0]), [a1] "+v"(a[h0 + 1]),
          [c00] "+v"(c[0][h0 + 0]), [c01] "+v"(c[0][h0 + 1]), [c10] "+v"(c[1][h0 + 0]),
          [c11] "+v"(c[1][h0 + 1]), [c20] "+v"(c[2][h0 + 0]), [c21] "+v"(c[2][h0 + 1])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [m2] "v"(m[2]),
          [q0] "s"(q[0]), [q1] "s"(q[1]));
  } else if constexpr (H == 2 && K == 4 && kFirst) {
    asm(POT_PAIR(POT_HEAD_K4, POT_DOT0, 0, 1)
        : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[h0 + 0]), [a1] "=&v"(a[h0 + 1]),
          [c00] "=&v"(c[0][h0 + 0]), [c01] "=&v"(c[0][h0 + 1]), [c10] "=&v"(c[1][h0 + 0]),
          [c11] "=&v"(c[1][h0 + 1]), [c20] "=&v"(c[2][h0 + 0]), [c21] "=&v"(c[2][h0 + 1]),
          [c30] "=&v"(c[3][h0 + 0]), [c31] "=&v"(c[3][h0 + 1])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [m2] "v"(m[2]),
          [m3] "v"(m[3]), [q0] "s"(q[0]), [q1] "s"(q[1]));
  } else if constexpr (H == 2 && K == 4 && !kFirst) {
    asm(POT_PAIR(POT_HEAD_K4, POT_DOTC, 0, 1)
        : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[h0 + 0]), [a1] "+v"(a[h0 + 1]),
          [c00] "+v"(c[0][h0 + 0]), [c01] "+v"(c[0][h0 + 1]), [c10] "+v"(c[1][h0 + 0]),
          [c11] "+v"(c[1][h0 + 1]), [c20] "+v"(c[2][h0 + 0]), [c21] "+v"(c[2][h0 + 1]),
          [c30] "+v"(c[3][h0 + 0]), [c31] "+v"(c[3][h0 + 1])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [m2] "v"(m[2]),
          [m3] "v"(m[3]), [q0] "s"(q[0]), [q1] "s"(q[1]));
  } else if constexpr (H == 4 && K == 2 && kFirst) {
    asm(POT_PAIR(POT_HEAD_K2, POT_DOT0, 0, 1) POT_PAIR(POT_HEAD_K2, POT_DOT0, 2, 3)
        : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[h0 + 0]), [a1] "=&v"(a[h0 + 1]),
          [a2] "=&v"(a[h0 + 2]), [a3] "=&v"(a[h0 + 3]), [c00] "=&v"(c[0][h0 + 0]),
          [c01] "=&v"(c[0][h0 + 1]), [c02] "=&v"(c[0][h0 + 2]), [c03] "=&v"(c[0][h0 + 3]),
          [c10] "=&v"(c[1][h0 + 0]), [c11] "=&v"(c[1][h0 + 1]), [c12] "=&v"(c[1][h0 + 2]),
          [c13] "=&v"(c[1][h0 + 3])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [q0] "s"(q[0]),
          [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]));
  } else if constexpr (H == 4 && K == 2 && !kFirst) {
    asm(POT_PAIR(POT_HEAD_K2, POT_DOTC, 0, 1) POT_PAIR(POT_HEAD_K2, POT_DOTC, 2, 3)
        : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[h0 + 0]), [a1] "+v"(a[h0 + 1]), [a2] "+v"(a[h0 + 2]),
          [a3] "+v"(a[h0 + 3]), [c00] "+v"(c[0][h0 + 0]), [c01] "+v"(c[0][h0 + 1]),
          [c02] "+v"(c[0][h0 + 2]), [c03] "+v"(c[0][h0 + 3]), [c10] "+v"(c[1][h0 + 0]),
          [c11] "+v"(c[1][h0 + 1]), [c12] "+v"(c[1][h0 + 2]), [c13] "+v"(c[1][h0 + 3])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [q0] "s"(q[0]),
          [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]));
  } else if constexpr (H == 4 && K == 3 && kFirst) {
    asm(POT_PAIR(POT_HEAD_K3, POT_DOT0, 0, 1) POT_PAIR(POT_HEAD_K3, POT_DOT0, 2, 3)
        : "=&v"(t0), "=&v"(t1), [a0] "=&v"(a[h0 + 0]), [a1] "=&v"(a[h0 + 1]),
          [a2] "=&v"(a[h0 + 2]), [a3] "=&v"(a[h0 + 3]), [c00] "=&v"(c[0][h0 + 0]),
          [c01] "=&v"(c[0][h0 + 1]), [c02] "=&v"(c[0][h0 + 2]), [c03] "=&v"(c[0][h0 + 3]),
          [c10] "=&v"(c[1][h0 + 0]), [c11] "=&v"(c[1][h0 + 1]), [c12] "=&v"(c[1][h0 + 2]),
          [c13] "=&v"(c[1][h0 + 3]), [c20] "=&v"(c[2][h0 + 0]), [c21] "=&v"(c[2][h0 + 1]),
          [c22] "=&v"(c[2][h0 + 2]), [c23] "=&v"(c[2][h0 + 3])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [m2] "v"(m[2]),
          [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]));
  } else if constexpr (H == 4 && K == 3 && !kFirst) {
    asm(POT_PAIR(POT_HEAD_K3, POT_DOTC, 0, 1) POT_PAIR(POT_HEAD_K3, POT_DOTC, 2, 3)
        : "=&v"(t0), "=&v"(t1), [a0] "+v"(a[h0 + 0]), [a1] "+v"(a[h0 + 1]), [a2] "+v"(a[h0 + 2]),
          [a3] "+v"(a[h0 + 3]), [c00] "+v"(c[0][h0 + 0]), [c01] "+v"(c[0][h0 + 1]),
          [c02] "+v"(c[0][h0 + 2]), [c03] "+v"(c[0][h0 + 3]), [c10] "+v"(c[1][h0 + 0]),
          [c11] "+v"(c[1][h0 + 1]), [c12] "+v"(c[1][h0 + 2]), [c13] "+v"(c[1][h0 + 3]),
          [c20] "+v"(c[2][h0 + 0]), [c21] "+v"(c[2][h0 + 1]), [c22] "+v"(c[2][h0 + 2]),
          [c23] "+v"(c[2][h0 + 3])
        : [sh] "v"(sh), [w] "v"(w), [m0] "v"(m[0]), [m1] "v"(m[1]), [m2] "v"(m[2]),
          [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]));
  }
}
#undef POT_PAIR
#undef POT_HEAD_K4
#undef POT_HEAD_K3
#undef POT_HEAD_K2
#undef POT_DOTC
#undef POT_DOT0
#undef POT_SAC_2
#undef POT_SAC_DC
#undef POT_SAC_D0
#undef POT_SAC_SH
typedef float float4v __attribute__((ext_vector_type(4)));

constexpr int kWaves = kBlock / 64;  // waves per workgroup of the default variant
// Waves per workgroup of the CU-wide variant (0: none). A SIMD issues the
// oldest of its ready waves first, so of the four equal workgroups that
// share a CU the first dispatched finishes in about a third of the time of
// the last, and the CU runs its last stretch with one wave per SIMD. In the
// CU-wide variant one workgroup holds all of a CU's waves (as many per SIMD
// as the kernel's registers allow: pool_waves) and its waves take tiles from
// a counter in LDS, so they all finish within about one tile of each other.
// Every engine but the fp16 comparator has it.
template <int MODE, int K, int VF>
constexpr int kPoolWaves = pool_waves(MODE, K, VF);
constexpr int kWTile = 64;    // keys per wave tile
constexpr int kXRow = 68;     // floats per head row of the transposed score tile
constexpr float kPScale = 12.0f;  // p is formed as 2^(x - M + 12) (fp16-normal range)
constexpr int kDppRowRor8 = 0x128;  // DPP row_ror:8: lane l reads lane l ^ 8 within its row of 16

// ---- VALU forms the compiler does not pick by itself ------------------------
__device__ __forceinline__ uint32_t xad_u32(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t r;
  asm("v_xad_u32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
// One 64-bit shift moves a pair of 32-bit words (v_lshrrev_b64 /
// v_lshlrev_b64 issue at the rate of a 32-bit shift).
__device__ __forceinline__ uint64_t pack64(uint32_t lo, uint32_t hi) {
  return ((uint64_t)hi << 32) | lo;
}
template <int S>
__device__ __forceinline__ uint64_t shr64(uint64_t v) {
  uint64_t r;
  asm("v_lshrrev_b64 %0, %1, %2" : "=v"(r) : "n"(S), "v"(v));
  return r;
}
template <int S>
__device__ __forceinline__ uint64_t shl64(uint64_t v) {
  uint64_t r;
  asm("v_lshlrev_b64 %0, %1, %2" : "=v"(r) : "n"(S), "v"(v));
  return r;
}

// Shift amounts and weight fields of the four element pairs of two PoT code
// words wa, wb (8 elements each; element m in nibble m = (sign << 3) | e).
// am[.][n]: the exponents of elements n and n + 4 in bits 3:0 and 19:16,
// where v_pk_ashrrev_i16 reads its per-half shift amounts (the bits above
// them in each half may be set: 20 and up hold bits of the other word).
// wf[.][n]: the weight field of elements n and n + 4, (sign, "not the zero
// code") in bits 15:14 and 31:30, so that an arithmetic shift of each half
// by 14 gives 1, -1, or 0 for the zero code (bits below 14 of each half are
// left as they come). The two words share every shift; sel must hold
// 0x88888888 (in a register, so that the select runs at the rate of a
// VGPR-only op).
struct CodePairFields {
  uint32_t am[2][4], wf[2][4];
};
__device__ __forceinline__ CodePairFields code_pair_fields(uint32_t wa, uint32_t wb,
                                                           uint32_t sel) {
  CodePairFields f;
  const uint32_t xa = wa & 0x77777777u, xb = wb & 0x77777777u;  // e per nibble
  // e + 1 per nibble (no carry between nibbles): bit 3 is set exactly for
  // the zero code, e = 7; moved to bit 2 by the pair's shift right by one
  const uint64_t ys = shr64<1>(pack64(xa + 0x11111111u, xb + 0x11111111u));
  // bit 3 of each nibble: the sign; bit 2: "not the zero code"
  const uint32_t swa = (wa & sel) | (~(uint32_t)ys & ~sel);
  const uint32_t swb = (wb & sel) | (~(uint32_t)(ys >> 32) & ~sel);
  const uint64_t xx = pack64(xa, xb);
  const uint64_t a1 = shr64<4>(xx), a2 = shr64<8>(xx), a3 = shr64<12>(xx);
  f.am[0][0] = xa;
  f.am[1][0] = xb;
  f.am[0][1] = (uint32_t)a1;
  f.am[1][1] = (uint32_t)(a1 >> 32);
  f.am[0][2] = (uint32_t)a2;
  f.am[1][2] = (uint32_t)(a2 >> 32);
  f.am[0][3] = (uint32_t)a3;
  f.am[1][3] = (uint32_t)(a3 >> 32);
  const uint64_t ss = pack64(swa, swb);
  const uint64_t s0 = shl64<12>(ss), s1 = shl64<8>(ss), s2 = shl64<4>(ss);
  f.wf[0][0] = (uint32_t)s0;
  f.wf[1][0] = (uint32_t)(s0 >> 32);
  f.wf[0][1] = (uint32_t)s1;
  f.wf[1][1] = (uint32_t)(s1 >> 32);
  f.wf[0][2] = (uint32_t)s2;
  f.wf[1][2] = (uint32_t)(s2 >> 32);
  f.wf[0][3] = swa;
  f.wf[1][3] = swb;
  return f;
}

// max(a, b) for scores (never NaN) as v_max_f32 without operand canonicalisation
__device__ __forceinline__ float max_f32(float a, float b) {
  return __builtin_amdgcn_fmed3f(a, b, __builtin_inff());
}


// Waits until this wave's vector stores are acknowledged by the L2. A
// workgroup barrier alone does not: it orders the wave's accesses for the
// other waves' vector loads, but the scalar cache, which reads the prepared
// query operands, fills from the L2.
__device__ __forceinline__ void wait_stores_in_l2() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---- streaming loads -----------------------------------------------------------
// The cache is read once per call, so its loads carry the non-temporal hint.
// It pays for the value fragments of every engine and for the 32-byte PoT
// code rows; the fp16 comparator's 128-byte key rows are read by eight
// 16-byte loads per lane that revisit the same lines, and stay plain there.
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));

// Raw buffer resources over the cache rows of one tile (gfx9 descriptor word
// 3 = 0x00020000: untyped records, byte-granular range). Each load's resource
// starts at the tile's first row and ends at the key range's last row, and
// the whole offset is in the vector operand: the hardware compares only that
// offset (not the scalar one) with the record count, so a lane whose key is
// at or past the end reads zeros and touches no memory. The tile loops need
// no clamped addresses, and every offset is 32-bit.
typedef __amdgpu_buffer_rsrc_t BufRsrc;
constexpr int kBufWord3 = 0x00020000;
constexpr int kAuxNt = 2;  // cache policy of the loads: non-temporal
__device__ __forceinline__ BufRsrc buf_rsrc(const void* base, int64_t n_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n_bytes,
                                           kBufWord3);
}

// The streams of one (batch, kv head) sequence that a workgroup reads, as
// byte pointers to the sequence's row 0 and the rows that exist: keys
// (codes, mantissa planes, scales) below t_end, value groups (fp16 or
// bytes, INT8 exponents) below v_end (the end of the range's last 8-key
// group).
struct Streams {
  const uint8_t* codes;
  const uint8_t* planes;
  const uint8_t* scales;
  const uint8_t* values;
  const uint8_t* exps;
  int t_end, v_end;
};

// Resource over rows t0 .. lim - 1 of row_bytes bytes each (t0 < lim, both
// wave-uniform, lim * row_bytes < 2^31).
__device__ __forceinline__ BufRsrc tile_rsrc(const uint8_t* base, int t0, int lim, int row_bytes) {
  return buf_rsrc(base + (uint32_t)(t0 * row_bytes), (int64_t)((lim - t0) * row_bytes));
}

// ---- per-tile register payloads -----------------------------------------------
template <int MODE, int K>
struct KeyRegs;
template <int K>
struct KeyRegs<kScorePot, K> {
  uint4 c0, c1;
  uint2 pl[K > 0 ? K : 1];
  float s;
};
template <int K>
struct KeyRegs<kScoreDs4a, K> {
  uint4 c0, c1;
  uint2 pl[K > 0 ? K : 1];
  float s;
};
template <int K>
struct KeyRegs<kScoreInt8, K> {
  int4 k[4];
  float s;
};
template <int K>
struct KeyRegs<kScoreFp16, K> {
  uint4 k[8];
};

template <bool V8>
struct ValRegs {
  uint4 f[2][4];  // [K-block of 32 keys][16-dim block], 8 fp16 values each
};
template <>
struct ValRegs<true> {
  uint2 f[2][4];  // the same fragments as 8 value bytes (v^ + 128)
  uint2 g;        // exponents g of the 8 keys whose weights this lane forms
};

// Loads are unconditional (addresses clamped into the valid range, or reads
// past a buffer resource's end, which return zeros) so that the compiler can
// count outstanding loads statically and keep the prefetch of the next tile in
// flight while the current one is processed; keys past the range are masked
// when the tile is consumed.
// Key rows of the comparators (INT8 codes, fp16 keys).
template <int MODE, int K>
__device__ __forceinline__ void load_keys(const DecodeArgs& a, int64_t row, KeyRegs<MODE, K>& r) {
  if constexpr (MODE == kScoreInt8) {
    const int4* kp = reinterpret_cast<const int4*>(a.codes_i8 + row * kDim);
#pragma unroll
    for (int i = 0; i < 4; ++i) r.k[i] = kp[i];
    r.s = a.key_scale[row];
  } else {
    const uint4* kp = reinterpret_cast<const uint4*>(a.k_f16 + row * kDim);
#pragma unroll
    for (int i = 0; i < 8; ++i) r.k[i] = kp[i];
  }
}

// PoT codes of keys t0 + lane (PoT and byte-decode engines): keys at or past
// the range's end read zeros (they are masked when the tile is consumed).
template <int MODE, int K>
__device__ __forceinline__ void load_keys_buf(const Streams& st, int t0, int lane,
                                              KeyRegs<MODE, K>& r) {
  const BufRsrc rc = tile_rsrc(st.codes, t0, st.t_end, kDim / 2);
  const u32x4v c0 = __builtin_amdgcn_raw_buffer_load_b128(rc, lane * 32, 0, kAuxNt);
  const u32x4v c1 = __builtin_amdgcn_raw_buffer_load_b128(rc, lane * 32 + 16, 0, kAuxNt);
  r.c0 = make_uint4(c0.x, c0.y, c0.z, c0.w);
  r.c1 = make_uint4(c1.x, c1.y, c1.z, c1.w);
  if constexpr (MODE == kScorePot || MODE == kScoreDs4a) {
    if constexpr (K > 0) {
      const BufRsrc rp = tile_rsrc(st.planes, t0, st.t_end, 8 * K);
#pragma unroll
      for (int bb = 0; bb < K; ++bb) {
        const u32x2v p = __builtin_amdgcn_raw_buffer_load_b64(rp, lane * 8 * K + 8 * bb, 0, kAuxNt);
        r.pl[bb] = make_uint2(p.x, p.y);
      }
    }
  }
  const BufRsrc rs = tile_rsrc(st.scales, t0, st.t_end, 4);
  r.s = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, lane * 4, 0, kAuxNt));
}

// B fragments of one 64-key tile: lane l takes keys t0 + 32*kb + 8*(l/16) ..+7
// of dim 16*nb + l%16, one 16-byte (fp16) or 8-byte (INT8) load each from the
// token-interleaved cache, through the tile's value resource: groups past
// the range's last group read zeros (their weights are 0). With INT8 values
// the lane also loads the exponents of the 8 keys t0 + 32*part + 8*grp ..+7
// whose weights it forms in stage 2.
template <bool V8>
__device__ __forceinline__ void load_values_buf(const Streams& st, int t0, int lane,
                                                ValRegs<V8>& v) {
  constexpr int kGroupBytes = V8 ? 8 * kDim : 16 * kDim;  // one 8-token group
  const BufRsrc rv = tile_rsrc(st.values, t0, st.v_end, kGroupBytes / 8);
  const int voff = (lane >> 4) * kGroupBytes + (lane & 15) * (V8 ? 8 : 16);
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int off = voff + kb * 4 * kGroupBytes + nb * 16 * (V8 ? 8 : 16);
      if constexpr (V8) {
        const u32x2v w = __builtin_amdgcn_raw_buffer_load_b64(rv, off, 0, kAuxNt);
        v.f[kb][nb] = make_uint2(w.x, w.y);
      } else {
        const u32x4v w = __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, kAuxNt);
        v.f[kb][nb] = make_uint4(w.x, w.y, w.z, w.w);
      }
    }
  }
  if constexpr (V8) {
    const int part = (lane & 15) >> 3, grp = lane >> 4;
    const BufRsrc re = tile_rsrc(st.exps, t0, st.v_end, 1);
    const u32x2v g = __builtin_amdgcn_raw_buffer_load_b64(re, 32 * part + 8 * grp, 0, 0);
    v.g = make_uint2(g.x, g.y);
  }
}

// fp16 B fragment of 8 INT8 values held as v^ + 128: bytes u become the fp16
// numbers 1024 + u = 1152 + v^ (bit pattern 0x6400 | u, exact), two per
// v_perm_b32; the 1152 offset is removed after accumulation with the weight
// sums.
__device__ __forceinline__ half8 int8_value_fragment(uint2 w) {
  constexpr uint32_t kHi = 0x64646464u;
  return __builtin_bit_cast(
      half8, make_uint4(__builtin_amdgcn_perm(kHi, w.x, 0x04010400u),
                        __builtin_amdgcn_perm(kHi, w.x, 0x04030402u),
                        __builtin_amdgcn_perm(kHi, w.y, 0x04010400u),
                        __builtin_amdgcn_perm(kHi, w.y, 0x04030402u)));
}
constexpr float kV8Offset = 1152.0f;

// Zero the value fragments of tokens at or past t_end (tail tile only), so
// that whatever the cache holds there cannot reach the sums (p is 0 there).
__device__ __forceinline__ void mask_values(int t0, int t_end, int lane, ValRegs<false>& v) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int g8 = t0 + 32 * kb + 8 * (lane >> 4);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      uint32_t w4[4] = {v.f[kb][nb].x, v.f[kb][nb].y, v.f[kb][nb].z, v.f[kb][nb].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t lo = (g8 + 2 * i < t_end) ? 0x0000FFFFu : 0u;
        const uint32_t hi = (g8 + 2 * i + 1 < t_end) ? 0xFFFF0000u : 0u;
        w4[i] &= lo | hi;
      }
      v.f[kb][nb] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
    }
  }
}

// ---- prepared query operands (workspace, one block per kv head) -------------
// PoT-4 and PoT-Mk: [(c * 4 + n) * G + h] = q 2^7 of elements 8c + n and
// 8c + n + 4 as signed 16-bit halves;
// PoT-Mk decoded to weights: the same words with q itself;
// INT8: [i * G + h] four int8 per word;
// byte decode: [(2c + o) * G + h] four int8 (elements 8c + o + 2t, t = 0..3);
// fp16: [i * G + h] two fp16 per word. The G per-head score factors follow.
template <int MODE, int G, int K>
struct QLayout {
  static constexpr int kCols = G;                              // one operand column per head
  static constexpr int kWords = (MODE == kScorePot || (MODE == kScoreDs4a && K > 0)) ? 32 * kCols
                                : (MODE == kScoreInt8 || MODE == kScoreDs4a) ? (kDim / 4) * G
                                                     : (kDim / 2) * G;
};

// The new token of one (batch, kv head) sequence appended at row T - 1
// (Sec. II-F, a cache that holds only codes): wave 0 encodes the key with the
// row absmax scale, wave 1 stores the values (fp16, or INT8 with their
// exponent). Only the workgroup whose key range holds row T - 1 calls it.
template <int K>
__device__ __forceinline__ void append_token(const DecodeArgs& a, int64_t seq, int wave) {
  const int64_t row = seq * a.t_cap + (a.T - 1);
  if (wave == 0)
    encode_key_row_wave<K>(reinterpret_cast<const __half*>(a.app_k) + seq * kDim, a.hadamard, 0,
                        a.app_key_scale + row, a.app_codes_se + row * (kDim / 2),
                        a.app_codes_m + row * 8 * K, a.app_tab);
  else if (wave == 1 && a.app_v8 != nullptr)
    store_value_token_i8_wave(a.app_v + seq * kDim, a.app_v8 + seq * a.t_cap * kDim,
                              a.app_v_exp + seq * a.t_cap, a.T - 1);
  else if (wave == 1)
    store_value_token_wave(a.app_v + seq * kDim, a.app_v_cache + seq * a.t_cap * kDim, a.T - 1);
}

// The query elements of the heads this wave prepares (wave w of NW: heads w,
// w + NW), one per lane; loaded first thing so that their latency overlaps
// the rest of the prologue.
template <int G, int NW>
struct QueryIn {
  static constexpr int kHeadsPerWave = (G + NW - 1) / NW;
  float v[kHeadsPerWave];
};
template <int G, int NW>
__device__ __forceinline__ QueryIn<G, NW> load_queries(const DecodeArgs& a, int kvh, int b) {
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  QueryIn<G, NW> qin;
#pragma unroll
  for (int i = 0; i < QueryIn<G, NW>::kHeadsPerWave; ++i) {
    const int h = wave + NW * i;
    qin.v[i] = h < G ? a.q[((int64_t)b * a.Hq + a.q_of_kv[kvh * G + h]) * kDim + lane] : 0.0f;
  }
  return qin;
}

// Rotates (optionally) and quantises the G query vectors of one (batch, kv
// head) and writes the operand words and per-head score factors that the
// score loop reads through the scalar cache, into qb (this workgroup's own
// slot of the workspace). Called by all NW waves of the workgroup; wave w
// handles heads w, w + NW, whose elements qin holds. taps: also write the q^
// and Delta debug taps.
template <int MODE, int G, int K, int NW>
__device__ __forceinline__ void prepare_queries(const DecodeArgs& a, int kvh, int b,
                                                int32_t* __restrict__ qb, bool taps,
                                                const QueryIn<G, NW>& qin) {
  using QL = QLayout<MODE, G, K>;
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  float* cb = reinterpret_cast<float*>(qb + QL::kWords);
  constexpr int kHeadsPerWave = QueryIn<G, NW>::kHeadsPerWave;
#pragma unroll
  for (int i = 0; i < kHeadsPerWave; ++i) {
    const int h = wave + NW * i;
    if (h >= G) break;
    const int64_t bq = (int64_t)b * a.Hq + a.q_of_kv[kvh * G + h];
    float qv = qin.v[i];
    if constexpr (MODE == kScoreFp16) {
      const uint32_t bits = __half_as_ushort(__float2half_rn(qv));
      const uint32_t other = __shfl_xor(bits, 1, 64);
      if ((lane & 1) == 0) qb[(lane >> 1) * G + h] = (int32_t)(bits | (other << 16));
      if (lane == 0) cb[h] = __fmul_rn(log2e_f32(), 0.125f);
    } else {
      if (a.hadamard) qv = (float)(wave_fwht64((double)qv) * 0.125);
      float step;
      const int qi = wave_quantize_int8(qv, &step);
      if constexpr (MODE == kScorePot || (MODE == kScoreDs4a && K > 0)) {
        // word ((c * 4 + n) * G + h) holds, for elements 8c + n (low half)
        // and 8c + n + 4 (high half), q 2^7 of head h: signed 16-bit
        // operands in [-16256, 16256] with 7 clear low bits, so an
        // arithmetic right shift by e <= 7 is exact. The decoded-weight
        // path takes q itself (its weights carry the 2^(7 - e)).
        constexpr int kMul = MODE == kScorePot ? 128 : 1;
        const uint32_t up = (uint32_t)__shfl_down(qi, 4, 64);
        if ((lane & 4) == 0)
          qb[((lane >> 3) * 4 + (lane & 3)) * G + h] =
              (int32_t)(((uint32_t)(qi * kMul) & 0xFFFFu) | ((up * (uint32_t)kMul) << 16));
        if (lane == 0)
          cb[h] = __fmul_rn(__fmul_rn(step, log2e_f32()),
                            __builtin_amdgcn_ldexpf(1.0f, -(a.frac_bits + K + 3)));
      } else if constexpr (MODE == kScoreDs4a) {
        // the word of code word c and parity o holds elements 8c + o + 2t in
        // byte t: lanes differing in bits 1 and 2 fill one word
        uint32_t word = (uint32_t)(qi & 0xFF) << (8 * ((lane >> 1) & 3));
        word |= __shfl_xor(word, 2, 64);
        word |= __shfl_xor(word, 4, 64);
        if ((lane & 6) == 0) qb[(2 * (lane >> 3) + (lane & 1)) * G + h] = (int32_t)word;
        if (lane == 0)
          cb[h] = __fmul_rn(__fmul_rn(step, log2e_f32()),
                            __builtin_amdgcn_ldexpf(1.0f, -(a.frac_bits + 3)));
      } else {
        uint32_t word = (uint32_t)(qi & 0xFF) << (8 * (lane & 3));
        word |= __shfl_xor(word, 1, 64);
        word |= __shfl_xor(word, 2, 64);
        if ((lane & 3) == 0) qb[(lane >> 2) * G + h] = (int32_t)word;
        if (lane == 0) cb[h] = __fmul_rn(__fmul_rn(step, log2e_f32()), 0.125f);
      }
      if (taps) {
        if (a.dbg_qhat) a.dbg_qhat[bq * kDim + lane] = (int8_t)qi;
        if (a.dbg_delta && lane == 0) a.dbg_delta[bq] = step;
      }
    }
  }
}

// ---- shared memory of the decode kernel -------------------------------------
template <int NW>
struct alignas(16) DecodeSmem {
  alignas(16) float x[NW][8][kXRow];  // transposed score tile per wave
  float wo[NW][16][kDim];             // per-wave P.V (rows: heads x {hi, lo})
  float wl[NW][16];
  float wp[NW][64];  // INT8 values: per-lane sums of the unscaled weights
  int wm[NW][8];
  int gm[NW];        // INT8 values: per-wave minimum exponent
  int next;          // CU-wide variant: the next unclaimed tile of the range
};

// VF: value format, 0 fp16 values, 1 INT8 values, 2 INT8 values with the
// power-of-two weights of eq. logsm.
// Resident waves per SIMD the register allocation must allow (1: no
// constraint). The decoded-weight PoT-Mk path and the one- and two-plane
// shift-accumulate paths would otherwise take a few registers more than four
// waves leave (three per SIMD); held to four they keep every value in
// registers, without spills (measured faster at every shape). The three-
// and four-plane paths run at two or three waves, where a tighter budget
// measured slower at B = 8.
template <int MODE, int K>
constexpr int kMinWaves = ((MODE == kScoreDs4a && K > 0) || (MODE == kScorePot && (K == 1 || K == 2)))
                              ? 4
                              : 1;

// NW: waves per workgroup, kWaves or kPoolWaves<MODE, K, VF> (the CU-wide
// variant, whose waves take their tiles from the counter sm.next).
template <int MODE, int G, int K, bool DEBUG, int VF, int NW>
// qbuf is passed on its own as a restrict parameter: the prepared query
// operands are never written here, which lets the compiler read them through
// the scalar cache even in the debug variants that store score taps.
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(
    NW > kWaves ? NW / 4 : kMinWaves<MODE, K>))) void decode_kernel(const DecodeArgs a,
                                                               const int32_t* __restrict__ qbuf) {
  using QL = QLayout<MODE, G, K>;
  constexpr bool kPool = NW > kWaves;
  constexpr int kBlk = 64 * NW;
  __shared__ DecodeSmem<NW> sm;
  constexpr bool V8 = VF != 0;
  constexpr bool kPow2 = VF == 2;
  constexpr int kCols = QL::kCols;

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is uniform in a wave; saying so keeps the tile loop's
  // control flow scalar (no per-lane loop exit masks)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int64_t seq = (int64_t)b * a.Hkv + kvh;
  const int64_t row0 = seq * a.t_cap;
  const int8_t* eseq = V8 ? a.v_exp + row0 : nullptr;
  // This workgroup's own slot of query operands and score factors: written
  // by the prologue below, then only read, through the scalar cache (which
  // starts each dispatch empty; no other workgroup touches the slot).
  const int64_t slot = seq * a.n_splits + split;
  const int32_t* __restrict__ qb = qbuf + slot * a.qstride;
  const float* __restrict__ cb = reinterpret_cast<const float*>(qb + QL::kWords);

  // ---- per-wave streaming over 64-key tiles ------------------------------------
  const int t_begin = split * a.split_len;
  const int t_end = min(a.T, t_begin + a.split_len);
  const int n_tiles = (t_end - t_begin + kWTile - 1) / kWTile;
  const int row = lane & 15, grp = lane >> 4, hrow = row & 7, part = row >> 3;
  const bool hvalid = hrow < G;

  const QueryIn<G, NW> qin = load_queries<G, NW>(a, kvh, b);
  // The sequence's new token (fused append) is written before any of this
  // workgroup's cache loads: only the workgroup whose range holds row T - 1
  // reads that row.
  if constexpr (MODE == kScorePot || MODE == kScoreDs4a) {
    if (a.app_k != nullptr && split == a.n_splits - 1) {  // uniform per workgroup
      append_token<K>(a, seq, wave);
      wait_stores_in_l2();
      __syncthreads();
    }
  }
  int gref = 0;
  float lsum = 0.0f;  // INT8 values: this lane's sum of the unscaled weights

  float4v acc[5];
#pragma unroll
  for (int nb = 0; nb < 5; ++nb) acc[nb] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
  int m_run = INT_MIN;
  half8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (_Float16)1.0f;
  // -1 kept opaque so that p - hi stays one fma_mix reading hi as fp16
  float neg_one = -1.0f;
  asm("" : "+v"(neg_one));
  // the sign-bit select of the code fields, kept in a VGPR (a VALU op that
  // reads an SGPR issues at the slower rate)
  uint32_t sign_sel = 0x88888888u;
  asm("" : "+v"(sign_sel));

  KeyRegs<MODE, K> kr[2];
  const int g_last = (t_end - 1) & ~7;  // first token of the range's last 8-token group
  Streams st{};
  st.t_end = t_end;
  st.v_end = g_last + 8;
  if constexpr (MODE == kScorePot || MODE == kScoreDs4a) {
    st.codes = a.codes_se + row0 * (kDim / 2);
    st.scales = reinterpret_cast<const uint8_t*>(a.key_scale + row0);
    if constexpr (K > 0) st.planes = a.codes_m + row0 * 8 * K;
  }
  if constexpr (V8) {
    st.values = a.v8 + row0 * kDim;
    st.exps = reinterpret_cast<const uint8_t*>(a.v_exp + row0);
  } else {
    st.values = reinterpret_cast<const uint8_t*>(a.v + row0 * kDim);
  }
  // key codes of tile jt; keys past the range read zeros (PoT, byte decode)
  // or the range's last key (INT8, fp16)
  auto load_keys_tile = [&](int jt, KeyRegs<MODE, K>& kk) {
    const int t0 = t_begin + kWTile * jt;
    if constexpr (MODE == kScorePot || MODE == kScoreDs4a)
      load_keys_buf<MODE, K>(st, t0, lane, kk);
    else
      load_keys<MODE, K>(a, row0 + min(t0 + lane, t_end - 1), kk);
  };
  // Tiles: wave w starts with tiles w and w + NW; after that the default
  // variant takes every NW-th tile and the CU-wide one claims the next
  // unclaimed tile (from 2 NW on) one tile ahead of its use.
  int j = wave;
  int jn = wave + NW;  // CU-wide variant: this wave's next tile
  int jc = 0;          // CU-wide variant: the tile claimed during the current one
  const int j_last = n_tiles - 1;
  if (j < n_tiles) load_keys_tile(j, kr[0]);
  if constexpr (kPool) {
    if (tid == 0) sm.next = 2 * NW;
  }

  // Query preparation into this workgroup's slot while the first codes load;
  // with INT8 values also the reference exponent g_ref = min g over this
  // workgroup's keys (Sec. II-E eq. av): weights are formed as p 2^(g_ref -
  // g_j) <= p, so they stay in fp16 range for any g, and the sums are scaled
  // by 2^-g_ref at the end (fp32). One barrier then publishes both.
  prepare_queries<MODE, G, K, NW>(a, kvh, b, a.qbuf + slot * a.qstride, DEBUG && split == 0,
                                  qin);
  if constexpr (V8) {
    int gmin = INT_MAX;
    for (int t = t_begin + 8 * tid; t < t_end; t += 8 * kBlk) {
      const uint2 w = *reinterpret_cast<const uint2*>(eseq + t);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int gi = (int)(int8_t)(((i < 4) ? w.x : w.y) >> (8 * (i & 3)));
        gmin = (t + i < t_end) ? min(gmin, gi) : gmin;
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) gmin = min(gmin, __shfl_xor(gmin, o, 64));
    if (lane == 0) sm.gm[wave] = gmin;
  }
  wait_stores_in_l2();
  __syncthreads();
  if constexpr (V8) {
    gref = sm.gm[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) gref = min(gref, sm.gm[w]);
  }
  // Fill the scalar cache with the slot's lines now, all at once (one load
  // per 64-byte line), instead of one miss per code word in the first tile.
  {
    uint32_t warm = 0;
#pragma unroll
    for (int l = 0; l < (QL::kWords + G + 15) / 16; ++l) warm ^= (uint32_t)qb[16 * l];
    asm volatile("" ::"s"(warm));
  }

  // PoT scoring is long enough to cover the latency of value loads issued at
  // the start of the tile; the short INT8 / fp16 scoring is not, so those
  // prefetch the values of this wave's next tile as well.
  constexpr bool kPrefetchV = !(MODE == kScorePot || (MODE == kScoreDs4a && K > 0));
  ValRegs<V8> vr[kPrefetchV ? 2 : 1];
  if constexpr (kPrefetchV) {
    if (j < n_tiles) load_values_buf<V8>(st, t_begin + kWTile * j, lane, vr[0]);
  }

  // Stage 1 of a tile: issue the loads it still needs and those of this
  // wave's next tile, score (the loads land meanwhile), transpose and find
  // the tile's integer maximum per head (returned in m_new).
  float xv[8];
  int m_new = m_run;
  auto stage1 = [&](const KeyRegs<MODE, K>& ks, KeyRegs<MODE, K>& knext, ValRegs<V8>& vs,
                    ValRegs<V8>& vnext, int jt) {
    const int t0 = t_begin + kWTile * jt;
    // the next tile's keys (past the range: the last tile again, unused)
    const int jl = min(kPool ? jn : jt + NW, j_last);
    if constexpr (kPrefetchV) {
      load_keys_tile(jl, knext);
      load_values_buf<V8>(st, t_begin + kWTile * jl, lane, vnext);
    } else {
      load_values_buf<V8>(st, t0, lane, vs);
      load_keys_tile(jl, knext);
    }
    if constexpr (kPool) {
      // claim the tile after jn now; it is needed one tile from now
      int c = 0;
      if (lane == 0) c = __hip_atomic_fetch_add(&sm.next, 1, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_WORKGROUP);
      jc = __builtin_amdgcn_readfirstlane(c);
    }
    const int t = t0 + lane;
    const bool kvalid = t < t_end;
    float xs[G];
    // ---- 1. scores (lane = key) ----
    // Query operands of the shift paths (two element pairs of every head per
    // chunk, 2 G words; 16 chunks per key): chunk c + 1 is requested
    // once chunk c is in registers, so every scalar load has a chunk's work to
    // land in (a wait on scalar loads covers all of them, as they may return
    // in any order). A zero offset that depends on the tile keeps the
    // compiler from hoisting the loads out of the loop, where 32 G words
    // would not fit in scalar registers.
    uint32_t qc[2][2 * kCols];
    auto load_chunk = [&](int c) {
      int toff = 0;
      asm("" : "+s"(toff) : "s"(jt));
#pragma unroll
      for (int k = 0; k < 2 * kCols; ++k) qc[c & 1][k] = (uint32_t)qb[toff + 2 * kCols * c + k];
    };
    // wait for chunk c, then request chunk c + 1
    auto next_chunk = [&](int c) {
      asm volatile("" ::"s"(qc[c & 1][0]), "s"(qc[c & 1][2 * kCols - 1]));
      __builtin_amdgcn_sched_barrier(0);
      if (c + 1 < 16) load_chunk(c + 1);
      __builtin_amdgcn_sched_barrier(0);
    };
    if constexpr (MODE == kScorePot) {
      const uint32_t w[8] = {ks.c0.x, ks.c0.y, ks.c0.z, ks.c0.w,
                             ks.c1.x, ks.c1.y, ks.c1.z, ks.c1.w};
      int32_t accv[G];
      // Two elements of one head per 16-bit-pair operand (element 8c + n in
      // the low half, 8c + n + 4 in the high half). v_pk_ashrrev_i16 shifts
      // each half by its element's exponent: q 2^7 >> e = q 2^(7 - e), exact.
      // v_dot2_i32_i16 (the dot unit's multiply-add) with weights sigma =
      // +-1 per half, and 0 for the zero code (e = 7, whose shifted operand
      // is q), then applies the signs and adds both halves into the int32
      // sum. PoT-Mk: the value is sigma (2^k + j)
      // 2^-e, so the key's sum is 2^k times the leading sum plus 2^b times
      // the sum over the elements whose mantissa j has bit b set, each over
      // the same shifted operands with weights sigma or 0.
      constexpr int KP = K > 0 ? K : 1;
      int32_t accm[KP][G];
      // With G > 1 the shifts and sums are assembly blocks per element pair
      // (sac_heads, sac_heads_m1, sac_heads_mk) over operand chunks (above).
      constexpr bool kRaw = G > 1;
      if constexpr (kRaw) load_chunk(0);
      // Shift amounts and weight fields: for PoT-4 and PoT-M1, two code words
      // at a time with the pair's 64-bit shifts (code_pair_fields); with two
      // or more mantissa planes, whose registers hold no second word's
      // fields, one word at a time: x holds
      // e per nibble, sw the sign in bit 3 and "not the zero code" in bit 2
      // (bit 3 of e + 1 is set exactly for e = 7; no carry between
      // nibbles), moved into place per element pair.
      constexpr bool kPairFields = K <= 1;
      CodePairFields pf;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        uint32_t x = 0, sw = 0;
        if constexpr (kPairFields) {
          if ((i & 1) == 0) pf = code_pair_fields(w[i], w[i + 1], sign_sel);
        } else {
          x = w[i] & 0x77777777u;
          sw = (w[i] & 0x88888888u) | (~((x + 0x11111111u) >> 1) & 0x44444444u);
        }
        // the mantissa bits of this code word's 8 elements, one byte per
        // plane, copied into both halves (bit n for element 8c + n in the
        // low half, bit n + 4 in the high half)
        uint32_t pb[KP];
#pragma unroll
        for (int bb = 0; bb < K; ++bb) {
          const uint32_t pw = (i < 4) ? ks.pl[bb].x : ks.pl[bb].y;
          pb[bb] = __builtin_amdgcn_perm(pw, pw, (uint32_t)(i & 3) * 0x00010001u | 0x0C000C00u);
        }
        // one head: this code word's four operand words, read as one scalar
        // group per tile (the zero offset as for the chunks)
        uint32_t qq[4 * kCols];
        if constexpr (!kRaw) {
          int toff = 0;
          asm("" : "+s"(toff) : "s"(jt));
#pragma unroll
          for (int k = 0; k < 4 * kCols; ++k) qq[k] = (uint32_t)qb[toff + 4 * kCols * i + k];
        }
#pragma unroll
        for (int n = 0; n < 4; ++n) {
          const int c = 2 * i + (n >> 1);  // operand chunk (kRaw)
          if constexpr (kRaw) {
            if ((n & 1) == 0) next_chunk(c);
          }
          // exponents of elements 8c + n and 8c + n + 4, one per half (the
          // shifts in sac_heads* read only the low four bits of each half, so
          // the bits above them stay; the one-head C++ path masks them)
          const uint32_t shr = kPairFields ? pf.am[i & 1][n] : x >> (4 * n);
          // the weights of elements 8c + n and 8c + n + 4
          const s16x2 sg =
              __builtin_bit_cast(s16x2, kPairFields ? pf.wf[i & 1][n] : sw << (12 - 4 * n)) >>
              (short)14;
          s16x2 mw[KP];
#pragma unroll
          for (int bb = 0; bb < K; ++bb) {
            // mantissa bit of each half moved to bit 15 and spread: the
            // plane's weight is sigma where the bit is set, else 0
            const u16x2 amt = {(unsigned short)(15 - n), (unsigned short)(11 - n)};
            const s16x2 bit =
                __builtin_bit_cast(s16x2, __builtin_bit_cast(u16x2, pb[bb]) << amt) >> (short)15;
            mw[bb] = bit & sg;
          }
          const bool first = i == 0 && n == 0;  // the first pair starts every sum from 0
          if constexpr (kRaw) {
            const uint32_t wsg = __builtin_bit_cast(uint32_t, sg);
            const uint32_t* qp = &qc[c & 1][kCols * (n & 1)];
            if constexpr (K == 0) {
              if (first)
                sac_heads<G, true>(accv, qp, shr, wsg);
              else
                sac_heads<G, false>(accv, qp, shr, wsg);
            } else if constexpr (K == 1) {
              const uint32_t wm = __builtin_bit_cast(uint32_t, mw[0]);
              if (first)
                sac_heads_m1<G, true>(accv, accm[0], qp, shr, wsg, wm);
              else
                sac_heads_m1<G, false>(accv, accm[0], qp, shr, wsg, wm);
            } else {
              constexpr int H = (K == 4 || G == 2) ? 2 : 4;
              uint32_t wm[K];
#pragma unroll
              for (int bb = 0; bb < K; ++bb) wm[bb] = __builtin_bit_cast(uint32_t, mw[bb]);
#pragma unroll
              for (int h0 = 0; h0 < G; h0 += H) {
                if (first)
                  sac_heads_mk<H, K, G, true>(accv, accm, h0, qp + h0, shr, wsg, wm);
                else
                  sac_heads_mk<H, K, G, false>(accv, accm, h0, qp + h0, shr, wsg, wm);
              }
            }
          } else {
            // one head: the same sums in C++ (with clamp set, |sum| <= 2 *
            // 16256 is never reached, the compiler emits the three-operand
            // form for the first pair instead of zeroing the sum first)
            const s16x2 pv = __builtin_bit_cast(s16x2, qq[n]) >>
                             __builtin_bit_cast(s16x2, shr & 0x000F000Fu);
            accv[0] = first ? __builtin_amdgcn_sdot2(pv, sg, 0, true)
                            : __builtin_amdgcn_sdot2(pv, sg, accv[0], false);
#pragma unroll
            for (int bb = 0; bb < K; ++bb)
              accm[bb][0] = first ? __builtin_amdgcn_sdot2(pv, mw[bb], 0, true)
                                  : __builtin_amdgcn_sdot2(pv, mw[bb], accm[bb][0], false);
          }
        }
      }
      if constexpr (K > 0) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          uint32_t t = (uint32_t)accv[h] << K;
#pragma unroll
          for (int bb = 0; bb < K; ++bb) t += (uint32_t)accm[bb][h] << bb;
          accv[h] = (int32_t)t;
        }
      }
      if (a.frac_bits != kFInt) {  // uniform: rescale to head-room F exactly
#pragma unroll
        for (int h = 0; h < G; ++h)
          accv[h] = a.frac_bits > kFInt
                        ? (int32_t)((uint32_t)accv[h] << (a.frac_bits - kFInt))
                        : (accv[h] >> (kFInt - a.frac_bits));
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const int32_t v = accv[h];
        xs[h] = __fmul_rn(__fmul_rn((float)v, ks.s), cb[h]);
        if constexpr (DEBUG) {
          if (a.dbg_scores && kvalid)
            a.dbg_scores[((int64_t)b * a.Hq + a.q_of_kv[kvh * G + h]) * a.T + t] = v;
        }
      }
    } else if constexpr (MODE == kScoreDs4a && K > 0) {
      // PoT-Mk codes decoded to 16-bit integer weights (a multiply path):
      // element m's weight is sigma (2^k + j) 2^(7 - e), 0 for the zero code,
      // at most 31 * 128 in magnitude; v_dot2_i32_i16 accumulates q^ times
      // the weights of two elements per head. The sum is exactly 2^k times
      // the key's sum of eq. sac at head-room 7 (eq. mant), the integer the
      // shift-accumulate path forms from its planes, with one dot per head
      // and element pair for any k.
      const uint32_t w[8] = {ks.c0.x, ks.c0.y, ks.c0.z, ks.c0.w,
                             ks.c1.x, ks.c1.y, ks.c1.z, ks.c1.w};
      int32_t accv[G];
      // the mantissas regrouped per element pair n: byte i of jw[n][hw]
      // holds j of element 8(4 hw + i) + n in bits 0..3 and of element
      // 8(4 hw + i) + n + 4 in bits 4..7 (bit m of plane byte i is bit b of
      // the mantissa of element 8i + m)
      uint32_t jw[4][2];
#pragma unroll
      for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int hw = 0; hw < 2; ++hw) {
          uint32_t jacc = 0;
#pragma unroll
          for (int bb = 0; bb < K; ++bb) {
            const uint32_t pw = hw ? ks.pl[bb].y : ks.pl[bb].x;
            const uint32_t t = (bb <= n) ? (pw >> (n - bb)) : (pw << (bb - n));
            jacc |= t & (0x11111111u << bb);
          }
          jw[n][hw] = jacc;
        }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t wi = w[i];
        const uint32_t x = wi & 0x77777777u;
        const uint32_t y = x + 0x11111111u;
        // per nibble, bit 3: the sign; bit 2: "not the zero code" (as in
        // the shift-accumulate path); ~wi holds 7 - e in each nibble's low
        // three bits
        const uint32_t sw = (wi & 0x88888888u) | (~(y >> 1) & 0x44444444u);
        const uint32_t nx = ~wi;
        // this code word's operands as one scalar group (one wait per code
        // word: the chunked loads of the shift paths measured slower here)
        int toff = 0;
        asm("" : "+s"(toff) : "s"(jt));
        uint32_t qq[4 * kCols];
#pragma unroll
        for (int k = 0; k < 4 * kCols; ++k) qq[k] = (uint32_t)qb[toff + 4 * kCols * i + k];
#pragma unroll
        for (int n = 0; n < 4; ++n) {
          // weights sigma 2^(7 - e) (0 for the zero code) of elements 8i + n
          // and 8i + n + 4, then times 2^k + j
          const s16x2 sg = __builtin_bit_cast(s16x2, sw << (12 - 4 * n)) >> (short)14;
          const s16x2 sh7 = __builtin_bit_cast(s16x2, (nx >> (4 * n)) & 0x00070007u);
          const u16x2 sgs = __builtin_bit_cast(u16x2, (s16x2)(sg << sh7));
          const uint32_t jb = __builtin_amdgcn_perm(jw[n][i >> 2], jw[n][i >> 2],
                                                    (uint32_t)(i & 3) * 0x00010001u | 0x0C000C00u);
          const u16x2 j4 = __builtin_bit_cast(u16x2, jb) >> u16x2{0, 4};
          const u16x2 jn = (j4 & u16x2{15, 15}) | u16x2{1 << K, 1 << K};
          const s16x2 wt = __builtin_bit_cast(s16x2, (u16x2)(jn * sgs));
#pragma unroll
          for (int h = 0; h < G; ++h) {
            const s16x2 qv = __builtin_bit_cast(s16x2, qq[kCols * n + h]);
            accv[h] = (i == 0 && n == 0) ? __builtin_amdgcn_sdot2(qv, wt, 0, true)
                                         : __builtin_amdgcn_sdot2(qv, wt, accv[h], false);
          }
        }
      }
      if (a.frac_bits != kFInt) {  // uniform: rescale to head-room F exactly
#pragma unroll
        for (int h = 0; h < G; ++h)
          accv[h] = a.frac_bits > kFInt
                        ? (int32_t)((uint32_t)accv[h] << (a.frac_bits - kFInt))
                        : (accv[h] >> (kFInt - a.frac_bits));
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const int32_t v = accv[h];
        xs[h] = __fmul_rn(__fmul_rn((float)v, ks.s), cb[h]);
        if constexpr (DEBUG) {
          if (a.dbg_scores && kvalid)
            a.dbg_scores[((int64_t)b * a.Hq + a.q_of_kv[kvh * G + h]) * a.T + t] = v;
        }
      }
    } else if constexpr (MODE == kScoreDs4a) {
      // Byte decode of the PoT-4 codes (the DS4A operation, eq. ds4a, in
      // software): a v_perm_b32 table maps each exponent field to 2^(6 - e)
      // (0 for the zero code), the sign is applied per byte as (m ^ N) + n
      // with N = 0xff and n = 1 in the bytes of negative elements (no carry
      // between bytes: m <= 64, and the zero code is never negative), and
      // v_dot4_i32_i8 accumulates q * sigma 2^(6 - e): the exact score at
      // head-room 6, which one left shift brings to F. A multiply path.
      const uint32_t w[8] = {ks.c0.x, ks.c0.y, ks.c0.z, ks.c0.w,
                             ks.c1.x, ks.c1.y, ks.c1.z, ks.c1.w};
      int32_t accd[G];
#pragma unroll
      for (int h = 0; h < G; ++h) accd[h] = 0;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint32_t wc = w[c];
        const uint32_t e0 = wc & 0x07070707u, e1 = (wc >> 4) & 0x07070707u;
        const uint32_t m0 = __builtin_amdgcn_perm(0x00010204u, 0x08102040u, e0);
        const uint32_t m1 = __builtin_amdgcn_perm(0x00010204u, 0x08102040u, e1);
        const uint32_t n0 = (wc >> 3) & 0x01010101u, n1 = (wc >> 7) & 0x01010101u;
        // 0xff in the bytes of negative elements as (n << 8) - n: the shift is
        // kept opaque, or the compiler forms n * 255 with the quarter-rate
        // v_mul_lo_u32
        uint32_t n0s = n0 << 8, n1s = n1 << 8;
        asm("" : "+v"(n0s), "+v"(n1s));
        const uint32_t k0 = xad_u32(m0, n0s - n0, n0);
        const uint32_t k1 = xad_u32(m1, n1s - n1, n1);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          accd[h] = __builtin_amdgcn_sdot4(qb[(2 * c) * G + h], (int32_t)k0, accd[h], false);
          accd[h] = __builtin_amdgcn_sdot4(qb[(2 * c + 1) * G + h], (int32_t)k1, accd[h], false);
        }
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const int32_t v = (int32_t)((uint32_t)accd[h] << (a.frac_bits - 6));
        xs[h] = __fmul_rn(__fmul_rn((float)v, ks.s), cb[h]);
        if constexpr (DEBUG) {
          if (a.dbg_scores && kvalid)
            a.dbg_scores[((int64_t)b * a.Hq + a.q_of_kv[kvh * G + h]) * a.T + t] = v;
        }
      }
    } else if constexpr (MODE == kScoreInt8) {
      int32_t kw[16];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        kw[4 * i] = ks.k[i].x;
        kw[4 * i + 1] = ks.k[i].y;
        kw[4 * i + 2] = ks.k[i].z;
        kw[4 * i + 3] = ks.k[i].w;
      }
      int32_t accd[G];
#pragma unroll
      for (int h = 0; h < G; ++h) accd[h] = 0;
#pragma unroll
      for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int h = 0; h < G; ++h)
          accd[h] = __builtin_amdgcn_sdot4(qb[i * G + h], kw[i], accd[h], false);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        xs[h] = __fmul_rn(__fmul_rn((float)accd[h], ks.s), cb[h]);
        if constexpr (DEBUG) {
          if (a.dbg_scores && kvalid)
            a.dbg_scores[((int64_t)b * a.Hq + a.q_of_kv[kvh * G + h]) * a.T + t] = accd[h];
        }
      }
    } else {
      uint32_t kw[32];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        kw[4 * i] = ks.k[i].x;
        kw[4 * i + 1] = ks.k[i].y;
        kw[4 * i + 2] = ks.k[i].z;
        kw[4 * i + 3] = ks.k[i].w;
      }
      float dot[G];
#pragma unroll
      for (int h = 0; h < G; ++h) dot[h] = 0.0f;
#pragma unroll
      for (int i = 0; i < 32; ++i)
#pragma unroll
        for (int h = 0; h < G; ++h)
          dot[h] = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, qb[i * G + h]),
                                          __builtin_bit_cast(half2v, kw[i]), dot[h], false);
#pragma unroll
      for (int h = 0; h < G; ++h) xs[h] = __fmul_rn(dot[h], cb[h]);
    }

    // ---- 2. transpose through wave-private LDS ----
    // Lane (row, grp) takes head row & 7 and keys 32 * part + 8 * grp .. + 7
    // of the tile (part = row >> 3), so every weight is computed once. Keys
    // past the range carry the score of the range's last key (clamped
    // loads) or of zero codes (buffer reads past the range): they are masked
    // below in the tail tile.
#pragma unroll
    for (int h = 0; h < G; ++h) sm.x[wave][h][lane] = xs[h];
    wave_sync_lds();
    {
      // rows of heads >= G are never written: read row 0 and discard
      const float4* src =
          reinterpret_cast<const float4*>(&sm.x[wave][hvalid ? hrow : 0][32 * part + 8 * grp]);
      const float4 u0 = src[0], u1 = src[1];
      const float r8[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) xv[i] = hvalid ? r8[i] : -INFINITY;
    }
    wave_sync_lds();  // the tile buffer is rewritten by the next tile
    const bool tail = t0 + kWTile > t_end;  // wave-uniform
    if (tail) {
      const int k0 = t0 + 32 * part + 8 * grp;
#pragma unroll
      for (int i = 0; i < 8; ++i) xv[i] = (k0 + i < t_end) ? xv[i] : -INFINITY;
      // weights past the range are 0; fp16 value bytes there could be inf or
      // NaN and are cleared, INT8 value bytes are always finite numbers
      if constexpr (!V8) mask_values(t0, t_end, lane, vs);
    }

    // ---- 3. integer running maximum per head ----
    float mx = xv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mx = max_f32(mx, xv[i]);
    mx = max_f32(mx, __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(
                                                   __builtin_bit_cast(int, mx), kDppRowRor8, 0xF,
                                                   0xF, true)));  // the other part
    // ceil is monotonic, so M = max over lanes of ceil(x): the reduction over
    // the four rows of 16 lanes runs on int32 (swap odd with even rows, then
    // the two halves; v_permlane*_swap, no LDS)
    // a lane whose keys are all past the range holds -inf (no int32 ceiling)
    int mt = (hvalid && mx > -INFINITY) ? (int)ceilf(mx) : INT_MIN;
    {
      const auto r16 = __builtin_amdgcn_permlane16_swap((uint32_t)mt, (uint32_t)mt, false, false);
      mt = max((int)r16[0], (int)r16[1]);
      const auto r32 = __builtin_amdgcn_permlane32_swap((uint32_t)mt, (uint32_t)mt, false, false);
      mt = max((int)r32[0], (int)r32[1]);
    }
    m_new = max(m_run, mt);
  };

  // acc <- diag(2^(M_old - M_new)) acc on the matrix cores: D = sum_j A_j B_j
  // with B_j = acc[.][j] (16x16x4 f32 layout: lane l holds row 4 (l / 16) + j
  // of column l % 16) and A_j[i][k] = f_i for i = 4k + j, else 0. Each
  // element gets one exact power-of-two product. It runs outside the hot
  // loop below, so the accumulators stay in the matrix-core registers there.
  auto rescale = [&]() {
    const float f = (m_run == INT_MIN) ? 0.0f : __builtin_amdgcn_ldexpf(1.0f, m_run - m_new);
    const int arow = lane & 15, acol = lane >> 4;
#pragma unroll
    for (int nb = 0; nb < 5; ++nb) {
      float4v d = float4v{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        d = __builtin_amdgcn_mfma_f32_16x16x4f32(arow == 4 * acol + jj ? f : 0.0f, acc[nb][jj], d,
                                                 0, 0, 0);
      acc[nb] = d;
    }
    if constexpr (V8) lsum *= f;
    m_run = m_new;
  };

  // Stage 2 of a tile: weights from the scores and P.V on the matrix cores.
  auto stage2 = [&](const ValRegs<V8>& vs) {
    // ---- 4. weights (fp16 high / low parts) and P.V on the matrix cores ----
    // Each lane splits its 8 weights into hi = rtz(p) and lo = rtz(p - hi)
    // and hands lo to its partner lane (row ^ 8). Block kb = 0 then takes
    // rows 0-7 = hi, 8-15 = lo of the part-0 weights; block kb = 1 takes rows
    // 0-7 = lo, 8-15 = hi of the part-1 weights. Rows h and h + 8 are summed
    // at the end, so both blocks see hi + lo of every weight.
    const float bias = hvalid ? kPScale - (float)m_run : 0.0f;
    uint32_t hw[4], lw[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float p0, p1;
      if constexpr (kPow2) {
        // A~ = 2^-k with k = M - ceil(x - 1/2) (M - x rounded half up):
        // p = 2^(ceil(x - 1/2) - M + 12), exact; keys masked to -inf get 0.
        // ceil(x - 1/2) is ceil(x), less one when ceil(x) - x >= 1/2: that
        // difference is exact in fp32 where it decides (x - 1/2 itself is
        // not: -0.5 + 2^-25 would round to -1)
        auto pw = [&](float x) -> float {
          const float c = ceilf(x);
          const float r = (c - x >= 0.5f) ? c - 1.0f : c;
          return x > -INFINITY
                     ? __builtin_amdgcn_ldexpf(1.0f, (int)r - m_run + (int)kPScale)
                     : 0.0f;
        };
        p0 = pw(xv[2 * i]);
        p1 = pw(xv[2 * i + 1]);
      } else {
        p0 = __builtin_amdgcn_exp2f(xv[2 * i] + bias);
        p1 = __builtin_amdgcn_exp2f(xv[2 * i + 1] + bias);
      }
      if constexpr (V8) {
        // the softmax sum takes p; A.V takes p 2^(g_ref - g) (exact scaling)
        lsum += p0;
        lsum += p1;
        const uint32_t gw = (i < 2) ? vs.g.x : vs.g.y;
        p0 = __builtin_amdgcn_ldexpf(p0, gref - (int)(int8_t)(gw >> (16 * (i & 1))));
        p1 = __builtin_amdgcn_ldexpf(p1, gref - (int)(int8_t)(gw >> (16 * (i & 1) + 8)));
      }
      const half2v hi = __builtin_bit_cast(half2v, __builtin_amdgcn_cvt_pkrtz(p0, p1));
      hw[i] = __builtin_bit_cast(uint32_t, hi);
      lw[i] = __builtin_bit_cast(
          uint32_t, __builtin_amdgcn_cvt_pkrtz(__builtin_fmaf(neg_one, (float)hi.x, p0),
                                               __builtin_fmaf(neg_one, (float)hi.y, p1)));
    }
    uint32_t a0w[4], a1w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t rl =
          (uint32_t)__builtin_amdgcn_mov_dpp((int)lw[i], kDppRowRor8, 0xF, 0xF, true);
      a0w[i] = part ? rl : hw[i];
      a1w[i] = part ? hw[i] : rl;
    }
    const half8 af0 = __builtin_bit_cast(half8, make_uint4(a0w[0], a0w[1], a0w[2], a0w[3]));
    const half8 af1 = __builtin_bit_cast(half8, make_uint4(a1w[0], a1w[1], a1w[2], a1w[3]));
    auto bfrag = [&](int kb, int nb) -> half8 {
      if constexpr (V8) return int8_value_fragment(vs.f[kb][nb]);
      else return __builtin_bit_cast(half8, vs.f[kb][nb]);
    };
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af0, bfrag(0, nb), acc[nb], 0, 0, 0);
    acc[4] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af0, ones, acc[4], 0, 0, 0);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af1, bfrag(1, nb), acc[nb], 0, 0, 0);
    acc[4] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af1, ones, acc[4], 0, 0, 0);
  };

  // The hot loop runs the tiles that do not raise any head's maximum; a tile
  // that does leaves it, is rescaled and finished in the outer loop (a few
  // times per wave). The prefetched registers move forward after each tile so
  // that every tile uses the same registers.
  auto advance = [&]() {
    kr[0] = kr[1];
    if constexpr (kPrefetchV) vr[0] = vr[1];
    if constexpr (kPool) {
      j = jn;
      jn = jc;
    } else {
      j += NW;
    }
  };
#pragma nounroll
  while (j < n_tiles) {
#pragma nounroll
    for (;;) {
      stage1(kr[0], kr[1], vr[0], vr[kPrefetchV ? 1 : 0], j);
      if (__any(m_new != m_run)) break;
      stage2(vr[0]);
      advance();
      if (j >= n_tiles) break;
    }
    if (j >= n_tiles) break;
    rescale();
    stage2(vr[0]);
    advance();
  }

  // ---- merge the four waves ---------------------------------------------------
#pragma unroll
  for (int r = 0; r < 4; ++r) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) sm.wo[wave][4 * grp + r][16 * nb + row] = acc[nb][r];
    if (row == 0) sm.wl[wave][4 * grp + r] = acc[4][r];
  }
  if (lane < 8) sm.wm[wave][lane] = m_run;
  if constexpr (V8) sm.wp[wave][lane] = lsum;
  __syncthreads();

  const int Sn = a.n_splits;
  for (int idx = tid; idx < G * kDim; idx += kBlk) {
    const int h = idx / kDim, d = idx % kDim;
    const int64_t bq = (int64_t)b * a.Hq + a.q_of_kv[kvh * G + h];
    int M = INT_MIN;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = max(M, sm.wm[w][h]);
    float o = 0.0f, l = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (sm.wm[w][h] == INT_MIN) continue;
      const float f = __builtin_amdgcn_ldexpf(1.0f, sm.wm[w][h] - M);
      if constexpr (V8) {
        // numerator sum w (1152 + v^) minus 1152 sum w; denominator sum p over
        // the 8 lanes that formed head h's weights
        const float num = (sm.wo[w][h][d] + sm.wo[w][h + 8][d]) -
                          kV8Offset * (sm.wl[w][h] + sm.wl[w][h + 8]);
        float lw = 0.0f;
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) lw += sm.wp[w][16 * gq + h] + sm.wp[w][16 * gq + h + 8];
        o = fmaf(f, num, o);
        l = fmaf(f, lw, l);
      } else {
        o = fmaf(f, sm.wo[w][h][d] + sm.wo[w][h + 8][d], o);
        l = fmaf(f, sm.wl[w][h] + sm.wl[w][h + 8], l);
      }
    }
    if constexpr (V8) o = __builtin_amdgcn_ldexpf(o, -gref);
    if (Sn == 1) {
      a.out[bq * kDim + d] = o / l;
      if constexpr (DEBUG) {
        if (d == 0 && a.dbg_m_final) a.dbg_m_final[bq] = M;
        if (d == 0 && a.dbg_m_split) a.dbg_m_split[bq] = M;
      }
    } else {
      const int64_t ps = bq * Sn + split;
      a.part_o[ps * kDim + d] = o;
      if (d == 0) {
        a.part_l[ps] = l;
        a.part_m[ps] = M;
        if constexpr (DEBUG) {
          if (a.dbg_m_split) a.dbg_m_split[ps] = M;
        }
      }
    }
  }
}

// Merges the key splits of one (batch, query head): M = max_s M_s and
// O = sum_s 2^(M_s - M) o_s / sum_s 2^(M_s - M) l_s with exact power-of-two
// weights (Sec. II-E). Grid B * Hq, 4 waves; wave w takes splits w, w + 4,
// ... with one lane per output dimension, and the four waves meet in LDS.
// Up to 64 splits, every load of a wave is issued before the first wait (one
// memory latency for the whole merge); more splits go through a loop.
constexpr int kCombineWaves = 4;
constexpr int kCombineBatch = 16;  // splits per wave in the single-batch path
template <bool DEBUG>
__global__ __launch_bounds__(64 * kCombineWaves) void combine_kernel(const DecodeArgs a) {
  __shared__ float so[kCombineWaves][kDim];
  __shared__ float sl[kCombineWaves];
  __shared__ int smax[kCombineWaves];
  const int64_t bq = blockIdx.x;
  const int tid = threadIdx.x, d = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int Sn = a.n_splits;
  const int32_t* __restrict__ pm = a.part_m + bq * Sn;
  const float* __restrict__ pl = a.part_l + bq * Sn;
  const float* __restrict__ po = a.part_o + bq * Sn * kDim;
  float L = 0.0f, O = 0.0f;
  int M;
  if (Sn <= kCombineWaves * kCombineBatch) {  // uniform
    // lane i (< 16) holds M_s and l_s of split s = w + 4 i; every lane holds
    // o_s[d] of all of them. Splits past the last read the last one
    // (unconditional loads, so all are in flight together) and are dropped.
    const int li = min(d, kCombineBatch - 1);
    const int s_l = w + kCombineWaves * li;
    const bool valid = d < kCombineBatch && s_l < Sn;
    const int m_l = pm[min(s_l, Sn - 1)];
    const float l_l = pl[min(s_l, Sn - 1)];
    float ov[kCombineBatch];
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i)
      ov[i] = po[min(w + kCombineWaves * i, Sn - 1) * kDim + d];
    int mw = valid ? m_l : INT_MIN;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mw = max(mw, __shfl_xor(mw, o, 64));
    if (d == 0) smax[w] = mw;
    __syncthreads();
    M = max(max(smax[0], smax[1]), max(smax[2], smax[3]));
    const float f_l = valid ? __builtin_amdgcn_ldexpf(1.0f, m_l - M) : 0.0f;
    float fl = f_l * l_l;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) fl += __shfl_xor(fl, o, 64);
    L = fl;
#pragma unroll
    for (int i = 0; i < kCombineBatch; ++i) {
      const float f = __builtin_bit_cast(
          float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, f_l), i));
      O = fmaf(f, ov[i], O);
    }
  } else {
    M = INT_MIN;
    for (int s = tid; s < Sn; s += 64 * kCombineWaves) M = max(M, pm[s]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) M = max(M, __shfl_xor(M, o, 64));
    if (d == 0) smax[w] = M;
    __syncthreads();
    M = max(max(smax[0], smax[1]), max(smax[2], smax[3]));
#pragma unroll 8
    for (int s = w; s < Sn; s += kCombineWaves) {
      const float f = __builtin_amdgcn_ldexpf(1.0f, pm[s] - M);
      L = fmaf(f, pl[s], L);
      O = fmaf(f, po[s * kDim + d], O);
    }
  }
  so[w][d] = O;
  if (d == 0) sl[w] = L;
  __syncthreads();
  if (w == 0) {
    O = so[0][d];
    L = sl[0];
#pragma unroll
    for (int i = 1; i < kCombineWaves; ++i) {
      O += so[i][d];
      L += sl[i];
    }
    a.out[bq * kDim + d] = O / L;
    if constexpr (DEBUG) {
      if (d == 0 && a.dbg_m_final) a.dbg_m_final[bq] = M;
    }
  }
}

template <int MODE, int G, int K, bool DEBUG, int VF>
static hipError_t launch_t(const DecodeArgs& a, hipStream_t stream, hipEvent_t ev_begin,
                           hipEvent_t ev_end) {
  if constexpr (VF != 0 && MODE != kScorePot && MODE != kScoreDs4a) {
    return hipErrorInvalidValue;
  } else {
  constexpr int PW = kPoolWaves<MODE, K, VF>;
  hipError_t e = hipSuccess;
  if (ev_begin != nullptr && (e = hipEventRecord(ev_begin, stream)) != hipSuccess) return e;
  const dim3 grid((uint32_t)a.n_splits, (uint32_t)a.Hkv, (uint32_t)a.B);
  if constexpr (PW > 0) {
    if (a.wg_waves == PW)
      hipLaunchKernelGGL((decode_kernel<MODE, G, K, DEBUG, VF, PW>), grid, dim3(64 * PW), 0,
                         stream, a, static_cast<const int32_t*>(a.qbuf));
    else
      hipLaunchKernelGGL((decode_kernel<MODE, G, K, DEBUG, VF, kWaves>), grid, dim3(kBlock), 0,
                         stream, a, static_cast<const int32_t*>(a.qbuf));
  } else {
    hipLaunchKernelGGL((decode_kernel<MODE, G, K, DEBUG, VF, kWaves>), grid, dim3(kBlock), 0,
                       stream, a, static_cast<const int32_t*>(a.qbuf));
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (ev_end != nullptr && (e = hipEventRecord(ev_end, stream)) != hipSuccess) return e;
  if (a.n_splits == 1) return hipSuccess;
  hipLaunchKernelGGL((combine_kernel<DEBUG>), dim3((uint32_t)(a.B * a.Hq)),
                     dim3(64 * kCombineWaves), 0, stream, a);
  return hipGetLastError();
  }
}

template <int MODE, int G, int K, int VF>
static int occupancy_t(bool pool) {
  constexpr int PW = kPoolWaves<MODE, K, VF>;
  int n = 0;
  hipError_t e;
  if constexpr (PW > 0) {
    if (pool)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &n, reinterpret_cast<const void*>(&decode_kernel<MODE, G, K, false, VF, PW>), 64 * PW,
          0);
    else
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &n, reinterpret_cast<const void*>(&decode_kernel<MODE, G, K, false, VF, kWaves>), kBlock,
          0);
  } else {
    if (pool) return 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &n, reinterpret_cast<const void*>(&decode_kernel<MODE, G, K, false, VF, kWaves>), kBlock, 0);
  }
  return e == hipSuccess ? n : 0;
}

template <int MODE, int G, bool DEBUG, int VF>
static hipError_t launch_k(int mant_bits, const DecodeArgs& a, hipStream_t stream, hipEvent_t e0,
                           hipEvent_t e1) {
  if constexpr (!(MODE == kScorePot || (MODE == kScoreDs4a && VF == 0))) {
    return launch_t<MODE, G, 0, DEBUG, VF>(a, stream, e0, e1);
  } else {
    switch (mant_bits) {
      case 0: return launch_t<MODE, G, 0, DEBUG, VF>(a, stream, e0, e1);
      case 1: return launch_t<MODE, G, 1, DEBUG, VF>(a, stream, e0, e1);
      case 2: return launch_t<MODE, G, 2, DEBUG, VF>(a, stream, e0, e1);
      case 3: return launch_t<MODE, G, 3, DEBUG, VF>(a, stream, e0, e1);
      case 4: return launch_t<MODE, G, 4, DEBUG, VF>(a, stream, e0, e1);
      default: return hipErrorInvalidValue;
    }
  }
}

template <int MODE, bool DEBUG, int VF>
static hipError_t launch_g(int G, int mant_bits, const DecodeArgs& a, hipStream_t stream,
                           hipEvent_t e0, hipEvent_t e1) {
  switch (G) {
    case 1: return launch_k<MODE, 1, DEBUG, VF>(mant_bits, a, stream, e0, e1);
    case 2: return launch_k<MODE, 2, DEBUG, VF>(mant_bits, a, stream, e0, e1);
    case 4: return launch_k<MODE, 4, DEBUG, VF>(mant_bits, a, stream, e0, e1);
    case 8: return launch_k<MODE, 8, DEBUG, VF>(mant_bits, a, stream, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

// One score mode and value format: every head-group size and mantissa width
// the mode supports (the instantiations live in one translation unit per
// mode / format, declared in pot_launch.hpp).
template <int MODE, int VF>
hipError_t launch_mode_vf(int G, int mant_bits, bool debug, const DecodeArgs& a,
                          hipStream_t stream, hipEvent_t e0, hipEvent_t e1) {
  if constexpr (MODE == kScoreFp16)
    return launch_g<MODE, false, VF>(G, mant_bits, a, stream, e0, e1);
  else
    return debug ? launch_g<MODE, true, VF>(G, mant_bits, a, stream, e0, e1)
                 : launch_g<MODE, false, VF>(G, mant_bits, a, stream, e0, e1);
}

template <int MODE, int VF>
int occupancy_mode_vf(int G, int mant_bits, bool pool) {
  auto by_k = [&](auto g_tag) -> int {
    constexpr int GG = decltype(g_tag)::value;
    if constexpr (MODE == kScorePot || (MODE == kScoreDs4a && VF == 0)) {
      switch (mant_bits) {
        case 0: return occupancy_t<MODE, GG, 0, VF>(pool);
        case 1: return occupancy_t<MODE, GG, 1, VF>(pool);
        case 2: return occupancy_t<MODE, GG, 2, VF>(pool);
        case 3: return occupancy_t<MODE, GG, 3, VF>(pool);
        default: return occupancy_t<MODE, GG, 4, VF>(pool);
      }
    } else {
      return occupancy_t<MODE, GG, 0, VF>(pool);
    }
  };
  switch (G) {
    case 1: return by_k(std::integral_constant<int, 1>{});
    case 2: return by_k(std::integral_constant<int, 2>{});
    case 4: return by_k(std::integral_constant<int, 4>{});
    default: return by_k(std::integral_constant<int, 8>{});
  }
}

}  // namespace potattn
