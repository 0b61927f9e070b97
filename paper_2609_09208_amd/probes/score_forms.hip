// Score-form probe: the exact int32 PoT-4 score of G = 8 query heads per key
// (Sec. II-B eq. sac, F = 7) in six gfx950 instruction forms, on the same
// codes and queries. One key per lane, codes streamed from HBM once; every
// form is checked against a host reference on the first 65536 keys, then
// timed over 4M keys (128 MiB of codes), where VALU issue binds.
//
//  0 sdwa     an earlier decode kernel core: two heads per 32-bit operand
//             Q2 = 2 (q_a + 2^16 q_b), SDWA v_lshlrev_b32 reading the shift
//             (6 - e) mod 32 from a byte, v_xad_u32 for the sign (ones'
//             complement, +1 per negative element from a popcount), 16-bit
//             fields unpacked by SDWA adds every 2 elements.
//  1 lshl_add v_lshl_add_u32 (shift and add in one): the sign must now be
//             applied before the shift (xor per head pair), the shift comes
//             from a VGPR (no byte select), and the ones' complement costs
//             -2^s per negative element in the low field, summed by one more
//             shift-add per element.
//  2 pk16     v_pk_lshrrev_b16 (the decode kernel's core before form 5):
//             two elements of one head per operand, (q + 128) 2^7 >> e =
//             (q + 128) 2^(7 - e) exactly (a right shift of an operand with 7
//             clear low bits), zero codes shifted by 15 to 0; v_dot2_i32_i16
//             with per-element weights +-1 applies the signs and accumulates
//             both halves; a ninth column with q = 0 removes the +128 bias.
//  3 ds4a     byte decode (v_perm_b32 table sigma 2^(6 - e)) and v_dot4_i32_i8
//             (the software packed shift-dot of eq. ds4a; a multiply path).
//  4 int8     v_dot4_i32_i8 on pre-decoded int8 codes (64 bytes per key): the
//             INT8 MAC baseline.
//  5 pk16s    signed operands q 2^7 shifted by v_pk_ashrrev_i16 (exact for
//             e <= 7), v_dot2_i32_i16 with weights 1 / -1 and 0 for the zero
//             code, formed per element as 4-bit nibbles by three v_bfi_b32 per
//             code word and sign-extended per half: no bias column (the
//             decode kernel's current core).
// Forms 3 and 4 produce the score at F = 6 and double it.
//
// Build and run on a gfx950 device:
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//         -o score_forms paper_2609_09208_amd/probes/score_forms.hip && ./score_forms
// ./score_forms --form F --reps R runs one form only (for counter runs).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
      exit(1);                                                                \
    }                                                                         \
  } while (0)

constexpr int kG = 8;
constexpr int kKeys = 1 << 22;
constexpr int kCheck = 1 << 16;
// operand words per form, one buffer read through the scalar cache
constexpr int kOffSdwa = 0;      // [code word i][32]: 4 steps x (4 pairs elem m, 4 pairs m+1)
constexpr int kOffPk = 256;      // [code word i][pair n][9]: 8 heads + the bias column
constexpr int kOffDs4a = 544;    // [(2c + o) * 8 + h]
constexpr int kOffInt8 = 672;    // [i * 8 + h], elements 4i .. 4i+3
constexpr int kOffPkS = 800;     // [code word i][pair n][8]: signed q 2^7 halves
constexpr int kOps = 1056;

typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// ---- form 0: SDWA shift + v_xad -------------------------------------------------
#define STEP8(JJ)                                                                          \
  "v_lshlrev_b32_sdwa %[p0], %[s0], %[a0] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_lshlrev_b32_sdwa %[p1], %[s0], %[a1] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_lshlrev_b32_sdwa %[p2], %[s0], %[a2] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_lshlrev_b32_sdwa %[p3], %[s0], %[a3] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_xad_u32 %[p0], %[p0], %[g0], %[bias]\n"                                              \
  "v_xad_u32 %[p1], %[p1], %[g0], %[bias]\n"                                              \
  "v_xad_u32 %[p2], %[p2], %[g0], %[bias]\n"                                              \
  "v_xad_u32 %[p3], %[p3], %[g0], %[bias]\n"                                              \
  "v_lshlrev_b32_sdwa %[t], %[s1], %[b0] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_xad_u32 %[p0], %[t], %[g1], %[p0]\n"                                                 \
  "v_lshlrev_b32_sdwa %[t], %[s1], %[b1] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_xad_u32 %[p1], %[t], %[g1], %[p1]\n"                                                 \
  "v_lshlrev_b32_sdwa %[t], %[s1], %[b2] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_xad_u32 %[p2], %[t], %[g1], %[p2]\n"                                                 \
  "v_lshlrev_b32_sdwa %[t], %[s1], %[b3] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_" #JJ \
  " src1_sel:DWORD\n"                                                                      \
  "v_xad_u32 %[p3], %[t], %[g1], %[p3]\n"                                                 \
  "v_add_u32_sdwa %[A0], %[p0], %[A0] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:DWORD\n" \
  "v_add_u32_sdwa %[B0], sext(%[p0]), %[B0] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:DWORD\n" \
  "v_add_u32_sdwa %[A1], %[p1], %[A1] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:DWORD\n" \
  "v_add_u32_sdwa %[B1], sext(%[p1]), %[B1] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:DWORD\n" \
  "v_add_u32_sdwa %[A2], %[p2], %[A2] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:DWORD\n" \
  "v_add_u32_sdwa %[B2], sext(%[p2]), %[B2] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:DWORD\n" \
  "v_add_u32_sdwa %[A3], %[p3], %[A3] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:DWORD\n" \
  "v_add_u32_sdwa %[B3], sext(%[p3]), %[B3] dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_1 src1_sel:DWORD"

template <int JJ>
__device__ __forceinline__ void sdwa_step(uint32_t s0, uint32_t s1, uint32_t g0, uint32_t g1,
                                          const uint32_t* qm, uint32_t (&A)[4],
                                          uint32_t (&B)[4]) {
  uint32_t p0, p1, p2, p3, t;
#define OPS                                                                                \
  : [p0] "=&v"(p0), [p1] "=&v"(p1), [p2] "=&v"(p2), [p3] "=&v"(p3), [t] "=&v"(t),         \
    [A0] "+v"(A[0]), [A1] "+v"(A[1]), [A2] "+v"(A[2]), [A3] "+v"(A[3]), [B0] "+v"(B[0]),   \
    [B1] "+v"(B[1]), [B2] "+v"(B[2]), [B3] "+v"(B[3])                                      \
  : [s0] "v"(s0), [s1] "v"(s1), [g0] "v"(g0), [g1] "v"(g1), [bias] "s"(0x8000u),           \
    [a0] "s"(qm[0]), [a1] "s"(qm[1]), [a2] "s"(qm[2]), [a3] "s"(qm[3]), [b0] "s"(qm[4]),    \
    [b1] "s"(qm[5]), [b2] "s"(qm[6]), [b3] "s"(qm[7])
  if constexpr (JJ == 0) asm(STEP8(0) OPS);
  else if constexpr (JJ == 1) asm(STEP8(1) OPS);
  else if constexpr (JJ == 2) asm(STEP8(2) OPS);
  else asm(STEP8(3) OPS);
#undef OPS
}

__device__ __forceinline__ void score_sdwa(const uint32_t (&w)[8], const uint32_t* __restrict__ q,
                                           int32_t (&acc)[kG]) {
  uint32_t A[4] = {0, 0, 0, 0}, B[4] = {0, 0, 0, 0};
  int nneg = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) nneg += __popc(w[i] & 0x88888888u);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t qq[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) qq[k] = q[kOffSdwa + 32 * i + k];
    const uint32_t s0 = 0x26262626u - (w[i] & 0x07070707u);
    const uint32_t s1 = 0x26262626u - ((w[i] >> 4) & 0x07070707u);
#define SG(JJ, o) (uint32_t)((int32_t)(w[i] << (28 - 8 * (JJ) - (o))) >> 31)
    sdwa_step<0>(s0, s1, SG(0, 0), SG(0, 4), qq + 0, A, B);
    sdwa_step<1>(s0, s1, SG(1, 0), SG(1, 4), qq + 8, A, B);
    sdwa_step<2>(s0, s1, SG(2, 0), SG(2, 4), qq + 16, A, B);
    sdwa_step<3>(s0, s1, SG(3, 0), SG(3, 4), qq + 24, A, B);
#undef SG
  }
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    acc[2 * p] = (int32_t)(A[p] - 32u * 0x8000u + (uint32_t)nneg);
    acc[2 * p + 1] = (int32_t)B[p];
  }
}

// ---- form 1: v_lshl_add_u32 -----------------------------------------------------
__device__ __forceinline__ uint32_t lshl_add(uint32_t a, uint32_t s, uint32_t c) {
  uint32_t r;
  asm("v_lshl_add_u32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(s), "v"(c));
  return r;
}

__device__ __forceinline__ void score_lshl_add(const uint32_t (&w)[8],
                                               const uint32_t* __restrict__ q,
                                               int32_t (&acc)[kG]) {
  uint32_t A[4] = {0, 0, 0, 0}, B[4] = {0, 0, 0, 0}, neg2s = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t qq[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) qq[k] = q[kOffSdwa + 32 * i + k];
    const uint32_t s0 = 0x26262626u - (w[i] & 0x07070707u);
    const uint32_t s1 = 0x26262626u - ((w[i] >> 4) & 0x07070707u);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const uint32_t sh0 = s0 >> (8 * jj), sh1 = s1 >> (8 * jj);  // shift uses bits 4:0
      const uint32_t g0 = (uint32_t)((int32_t)(w[i] << (28 - 8 * jj)) >> 31);
      const uint32_t g1 = (uint32_t)((int32_t)(w[i] << (24 - 8 * jj)) >> 31);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        uint32_t P = lshl_add(qq[8 * jj + p] ^ g0, sh0, 0x8000u);
        P = lshl_add(qq[8 * jj + 4 + p] ^ g1, sh1, P);
        A[p] += P & 0xFFFFu;
        B[p] += (uint32_t)((int32_t)P >> 16);
      }
      // (~Q2) << s = -(Q2 << s) - 2^s: -2^s per negative element lands in
      // the low field; the shift-add of the sign word sums it
      neg2s = lshl_add(g0, sh0, neg2s);
      neg2s = lshl_add(g1, sh1, neg2s);
    }
  }
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    acc[2 * p] = (int32_t)(A[p] - 32u * 0x8000u - neg2s);
    acc[2 * p + 1] = (int32_t)B[p];
  }
}

// ---- form 2: v_pk_lshrrev_b16 + v_dot2_i32_i16 -----------------------------------
__device__ __forceinline__ void score_pk16(const uint32_t (&w)[8], const uint32_t* __restrict__ q,
                                           int32_t (&acc)[kG]) {
  int32_t a9[kG + 1];
#pragma unroll
  for (int h = 0; h <= kG; ++h) a9[h] = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t wi = w[i];
    // zero code (e = 7) -> shift 15; e keeps its value otherwise
    const uint32_t z = wi & (wi >> 1) & (wi >> 2) & 0x11111111u;
    const uint32_t x = (wi & 0x77777777u) | (z << 3);
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const u16x2 sh = __builtin_bit_cast(u16x2, x >> (4 * n));
      const s16x2 sg16 = __builtin_bit_cast(s16x2, wi << (12 - 4 * n)) >> (short)15;
      const s16x2 sg = __builtin_bit_cast(s16x2, __builtin_bit_cast(uint32_t, sg16) | 0x00010001u);
#pragma unroll
      for (int h = 0; h <= kG; ++h) {
        const u16x2 qb = __builtin_bit_cast(u16x2, q[kOffPk + 36 * i + 9 * n + h]);
        const u16x2 p = qb >> (sh & (unsigned short)15);
        a9[h] = __builtin_amdgcn_sdot2(__builtin_bit_cast(s16x2, p), sg, a9[h], false);
      }
    }
  }
#pragma unroll
  for (int h = 0; h < kG; ++h) acc[h] = a9[h] - a9[kG];
}

// ---- form 5: signed v_pk_ashrrev_i16 + v_dot2_i32_i16, weights 1 / 0 / -1 ----------
__device__ __forceinline__ uint32_t bfi_u32(uint32_t m, uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(m), "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ void score_pk16s(const uint32_t (&w)[8], const uint32_t* __restrict__ q,
                                            int32_t (&acc)[kG]) {
#pragma unroll
  for (int h = 0; h < kG; ++h) acc[h] = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t wi = w[i];
    // weight nibble: bit 0 = (e != 7), bits 1..3 = the sign bit
    const uint32_t s1 = wi >> 1, s2 = wi >> 2;
    const uint32_t sw =
        bfi_u32(0x77777777u, bfi_u32(0x33333333u, bfi_u32(0x11111111u, ~(wi & s1 & s2), s2), s1), wi);
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const s16x2 sh = __builtin_bit_cast(s16x2, (wi >> (4 * n)) & 0x00070007u);
      const s16x2 sg = __builtin_bit_cast(s16x2, sw << (12 - 4 * n)) >> (short)12;
#pragma unroll
      for (int h = 0; h < kG; ++h) {
        const s16x2 p = __builtin_bit_cast(s16x2, q[kOffPkS + 32 * i + 8 * n + h]) >> sh;
        acc[h] = __builtin_amdgcn_sdot2(p, sg, acc[h], false);
      }
    }
  }
}

// ---- form 3: byte decode + v_dot4 (software DS4A) ---------------------------------
__device__ __forceinline__ void score_ds4a(const uint32_t (&w)[8], const uint32_t* __restrict__ q,
                                           int32_t (&acc)[kG]) {
  int32_t d[kG];
#pragma unroll
  for (int h = 0; h < kG; ++h) d[h] = 0;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const uint32_t wc = w[c];
    const uint32_t m0 = __builtin_amdgcn_perm(0x00010204u, 0x08102040u, wc & 0x07070707u);
    const uint32_t m1 = __builtin_amdgcn_perm(0x00010204u, 0x08102040u, (wc >> 4) & 0x07070707u);
    const uint32_t n0 = (wc >> 3) & 0x01010101u, n1 = (wc >> 7) & 0x01010101u;
    const uint32_t k0 = (m0 ^ ((n0 << 8) - n0)) + n0, k1 = (m1 ^ ((n1 << 8) - n1)) + n1;
#pragma unroll
    for (int h = 0; h < kG; ++h) {
      d[h] = __builtin_amdgcn_sdot4(q[kOffDs4a + (2 * c) * kG + h], (int32_t)k0, d[h], false);
      d[h] = __builtin_amdgcn_sdot4(q[kOffDs4a + (2 * c + 1) * kG + h], (int32_t)k1, d[h], false);
    }
  }
#pragma unroll
  for (int h = 0; h < kG; ++h) acc[h] = 2 * d[h];
}

// ---- form 4: INT8 codes + v_dot4 ----------------------------------------------------
__device__ __forceinline__ void score_int8(const uint4 (&k)[4], const uint32_t* __restrict__ q,
                                           int32_t (&acc)[kG]) {
  const uint32_t kw[16] = {k[0].x, k[0].y, k[0].z, k[0].w, k[1].x, k[1].y, k[1].z, k[1].w,
                           k[2].x, k[2].y, k[2].z, k[2].w, k[3].x, k[3].y, k[3].z, k[3].w};
  int32_t d[kG];
#pragma unroll
  for (int h = 0; h < kG; ++h) d[h] = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i)
#pragma unroll
    for (int h = 0; h < kG; ++h)
      d[h] = __builtin_amdgcn_sdot4(q[kOffInt8 + i * kG + h], (int32_t)kw[i], d[h], false);
#pragma unroll
  for (int h = 0; h < kG; ++h) acc[h] = 2 * d[h];
}

template <int FORM>
__global__ __launch_bounds__(256) void k_score(const uint4* __restrict__ codes,
                                               const uint4* __restrict__ codes8,
                                               const uint32_t* __restrict__ q, int n,
                                               int32_t* __restrict__ scores,
                                               uint32_t* __restrict__ sums) {
  int it = 0;
  for (int key = blockIdx.x * 256 + threadIdx.x; key < n; key += gridDim.x * 256, ++it) {
    // the operands are re-read for every key, as the decode kernel re-reads
    // them for every tile: a zero offset that depends on the iteration keeps
    // the compiler from hoisting all of them into registers (which would not
    // fit and would spill into vector-register lanes)
    int off = 0;
    asm("" : "+s"(off) : "s"(it));
    const uint32_t* __restrict__ qk = q + off;
    int32_t acc[kG];
    if constexpr (FORM == 4) {
      uint4 k[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) k[j] = codes8[4 * key + j];
      score_int8(k, qk, acc);
    } else {
      const uint4 c0 = codes[2 * key], c1 = codes[2 * key + 1];
      const uint32_t w[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
      if constexpr (FORM == 0) score_sdwa(w, qk, acc);
      if constexpr (FORM == 1) score_lshl_add(w, qk, acc);
      if constexpr (FORM == 2) score_pk16(w, qk, acc);
      if constexpr (FORM == 3) score_ds4a(w, qk, acc);
      if constexpr (FORM == 5) score_pk16s(w, qk, acc);
    }
    uint32_t s = 0;
#pragma unroll
    for (int h = 0; h < kG; ++h) s += (uint32_t)acc[h] * (2u * h + 1u);
    sums[key] = s;
    if (scores != nullptr)
#pragma unroll
      for (int h = 0; h < kG; ++h) scores[(int64_t)key * kG + h] = acc[h];
  }
}

typedef void (*KernelFn)(const uint4*, const uint4*, const uint32_t*, int, int32_t*, uint32_t*);
static const KernelFn kForms[6] = {k_score<0>, k_score<1>, k_score<2>,
                                   k_score<3>, k_score<4>, k_score<5>};
static const char* kNames[6] = {"sdwa", "lshl_add", "pk16 + dot2 (bias column)",
                                "ds4a byte decode + dot4", "int8 dot4 (64 B/key)",
                                "pk16s signed + dot2"};

static uint64_t g_rng = 0x9E3779B97F4A7C15ull;
static uint32_t rnd() {
  g_rng = g_rng * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(g_rng >> 33);
}

int main(int argc, char** argv) {
  int only = -1, reps = 10;
  for (int a = 1; a + 1 < argc; a += 2) {
    if (!strcmp(argv[a], "--form")) only = atoi(argv[a + 1]);
    if (!strcmp(argv[a], "--reps")) reps = atoi(argv[a + 1]);
  }
  // codes: nibble (neg << 3) | e, e uniform in 0..7, 7 = zero with neg = 0
  std::vector<uint32_t> codes((size_t)kKeys * 8);
  std::vector<int8_t> codes8((size_t)kKeys * 64);
  std::vector<int> nib(64);
  for (int k = 0; k < kKeys; ++k) {
    for (int m = 0; m < 64; ++m) {
      const int e = rnd() % 8, neg = (e == 7) ? 0 : (int)(rnd() & 1);
      nib[m] = (neg << 3) | e;
      codes8[(size_t)k * 64 + m] = (int8_t)(e == 7 ? 0 : (neg ? -1 : 1) * (1 << (6 - e)));
    }
    for (int i = 0; i < 8; ++i) {
      uint32_t wv = 0;
      for (int t = 0; t < 8; ++t) wv |= (uint32_t)nib[8 * i + t] << (4 * t);
      codes[(size_t)k * 8 + i] = wv;
    }
  }
  int qh[kG][64];
  for (int h = 0; h < kG; ++h)
    for (int m = 0; m < 64; ++m) qh[h][m] = (int)(rnd() % 255) - 127;
  std::vector<uint32_t> ops(kOps, 0);
  for (int i = 0; i < 8; ++i)
    for (int jj = 0; jj < 4; ++jj)
      for (int p = 0; p < 4; ++p) {
        for (int o = 0; o < 2; ++o) {
          const int m = 8 * i + 2 * jj + o;
          ops[kOffSdwa + 32 * i + 8 * jj + 4 * o + p] =
              ((uint32_t)qh[2 * p][m] + ((uint32_t)qh[2 * p + 1][m] << 16)) << 1;
        }
      }
  for (int i = 0; i < 8; ++i)
    for (int n = 0; n < 4; ++n)
      for (int h = 0; h <= kG; ++h) {
        auto qb = [&](int m) { return (uint32_t)((h < kG ? qh[h][m] : 0) + 128) << 7; };
        ops[kOffPk + 36 * i + 9 * n + h] = qb(8 * i + n) | (qb(8 * i + n + 4) << 16);
      }
  for (int i = 0; i < 8; ++i)
    for (int n = 0; n < 4; ++n)
      for (int h = 0; h < kG; ++h) {
        auto qs = [&](int m) { return (uint32_t)(qh[h][m] * 128) & 0xFFFFu; };
        ops[kOffPkS + 32 * i + 8 * n + h] = qs(8 * i + n) | (qs(8 * i + n + 4) << 16);
      }
  for (int c = 0; c < 8; ++c)
    for (int o = 0; o < 2; ++o)
      for (int h = 0; h < kG; ++h) {
        uint32_t wv = 0;
        for (int t = 0; t < 4; ++t) wv |= (uint32_t)(uint8_t)qh[h][8 * c + o + 2 * t] << (8 * t);
        ops[kOffDs4a + (2 * c + o) * kG + h] = wv;
      }
  for (int i = 0; i < 16; ++i)
    for (int h = 0; h < kG; ++h) {
      uint32_t wv = 0;
      for (int t = 0; t < 4; ++t) wv |= (uint32_t)(uint8_t)qh[h][4 * i + t] << (8 * t);
      ops[kOffInt8 + i * kG + h] = wv;
    }
  // host reference: sum of sigma q 2^(7 - e) over non-zero codes
  std::vector<int32_t> ref((size_t)kCheck * kG);
  for (int k = 0; k < kCheck; ++k)
    for (int h = 0; h < kG; ++h) {
      int64_t s = 0;
      for (int m = 0; m < 64; ++m) {
        const int nb = (codes[(size_t)k * 8 + m / 8] >> (4 * (m % 8))) & 15, e = nb & 7;
        if (e == 7) continue;
        s += (int64_t)((nb & 8) ? -1 : 1) * qh[h][m] * (1 << (7 - e));
      }
      ref[(size_t)k * kG + h] = (int32_t)s;
    }

  uint4 *d_codes, *d_codes8;
  uint32_t *d_ops, *d_sums;
  int32_t* d_scores;
  CHECK(hipMalloc(&d_codes, codes.size() * 4));
  CHECK(hipMalloc(&d_codes8, codes8.size()));
  CHECK(hipMalloc(&d_ops, kOps * 4));
  CHECK(hipMalloc(&d_sums, (size_t)kKeys * 4));
  CHECK(hipMalloc(&d_scores, (size_t)kCheck * kG * 4));
  CHECK(hipMemcpy(d_codes, codes.data(), codes.size() * 4, hipMemcpyHostToDevice));
  CHECK(hipMemcpy(d_codes8, codes8.data(), codes8.size(), hipMemcpyHostToDevice));
  CHECK(hipMemcpy(d_ops, ops.data(), kOps * 4, hipMemcpyHostToDevice));
  int cus = 0;
  CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  std::vector<int32_t> got((size_t)kCheck * kG);
  printf("%-26s %10s %10s %12s %8s\n", "form", "best us", "median us", "keys/ns", "check");
  for (int f = 0; f < 6; ++f) {
    if (only >= 0 && f != only) continue;
    const dim3 grid_chk(kCheck / 256), grid(cus * 8);
    hipLaunchKernelGGL(kForms[f], grid_chk, dim3(256), 0, 0, d_codes, d_codes8, d_ops, kCheck,
                       d_scores, d_sums);
    CHECK(hipGetLastError());
    CHECK(hipMemcpy(got.data(), d_scores, got.size() * 4, hipMemcpyDeviceToHost));
    size_t bad = 0;
    for (size_t i = 0; i < got.size(); ++i) bad += got[i] != ref[i];
    std::vector<float> ms;
    for (int r = 0; r < reps + 2; ++r) {
      CHECK(hipEventRecord(e0, 0));
      hipLaunchKernelGGL(kForms[f], grid, dim3(256), 0, 0, d_codes, d_codes8, d_ops, kKeys,
                         nullptr, d_sums);
      CHECK(hipEventRecord(e1, 0));
      CHECK(hipEventSynchronize(e1));
      float t = 0;
      CHECK(hipEventElapsedTime(&t, e0, e1));
      if (r >= 2) ms.push_back(t);
    }
    CHECK(hipGetLastError());
    std::sort(ms.begin(), ms.end());
    const float best = ms.front() * 1e3f, med = ms[ms.size() / 2] * 1e3f;
    printf("%-26s %10.1f %10.1f %12.2f %8s\n", kNames[f], best, med, kKeys / (med * 1e3f),
           bad ? "FAIL" : "ok");
    if (bad) {
      fprintf(stderr, "form %d: %zu of %zu scores differ from the reference\n", f, bad,
              got.size());
      return 2;
    }
  }
  CHECK(hipFree(d_codes));
  CHECK(hipFree(d_codes8));
  CHECK(hipFree(d_ops));
  CHECK(hipFree(d_sums));
  CHECK(hipFree(d_scores));
  return 0;
}
