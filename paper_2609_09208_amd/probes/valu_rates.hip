// Issue-rate probe for the gfx950 VALU instruction forms the decode kernels use.
//
// Each kernel runs N iterations over 8 register chains of one instruction form
// (inline assembly, so the form is exactly the one named); only registers are
// touched, and each thread writes one word of a buffer sized to the grid.
// Reported: wave64 instructions per nanosecond per CU (2.4 per ns = one per
// cycle per CU at 2.4 GHz).
//
// Build and run on a gfx950 device:
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//         -o valu_rates paper_2609_09208_amd/probes/valu_rates.hip && ./valu_rates
#include <hip/hip_runtime.h>

#include <cstdio>

#define N 4096
#define BODY8(INS) INS(a0) INS(a1) INS(a2) INS(a3) INS(a4) INS(a5) INS(a6) INS(a7)
#define KERNEL(NAME, INS)                                                                 \
  __global__ __launch_bounds__(256) void NAME(unsigned* out, unsigned s, unsigned sh) {    \
    unsigned a0 = threadIdx.x, a1 = a0 + 1, a2 = a0 + 2, a3 = a0 + 3, a4 = a0 + 4,       \
             a5 = a0 + 5, a6 = a0 + 6, a7 = a0 + 7, b = a0 * 3u + 1u, c = sh;             \
    for (int i = 0; i < N; ++i) {                                                          \
      BODY8(INS)                                                                           \
    }                                                                                      \
    out[blockIdx.x * 256 + threadIdx.x] = a0 ^ a1 ^ a2 ^ a3 ^ a4 ^ a5 ^ a6 ^ a7 ^ b ^ c;   \
  }

#define I_ADD(x) asm volatile("v_add_u32_e32 %0, %1, %0" : "+v"(x) : "v"(b));
#define I_ADD_SGPR(x) asm volatile("v_add_u32_e32 %0, %1, %0" : "+v"(x) : "s"(s));
#define I_ADD_E64(x) asm volatile("v_add_u32_e64 %0, %1, %0" : "+v"(x) : "v"(b));
#define I_XOR(x) asm volatile("v_xor_b32_e32 %0, %1, %0" : "+v"(x) : "v"(b));
#define I_AND_LIT(x) asm volatile("v_and_b32_e32 %0, 0x7070707, %0" : "+v"(x));
#define I_MUL_F32(x) asm volatile("v_mul_f32_e32 %0, %1, %0" : "+v"(x) : "v"(b));
#define I_FMA_F32(x) asm volatile("v_fma_f32 %0, %1, %2, %0" : "+v"(x) : "v"(b), "v"(c));
#define I_LSHL(x) asm volatile("v_lshlrev_b32_e32 %0, %1, %0" : "+v"(x) : "v"(c));
#define I_LSHL_SDWA(x)                                                                       \
  asm volatile("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD "         \
               "src0_sel:BYTE_1 src1_sel:DWORD" : "=v"(x) : "v"(c), "s"(s));
#define I_ADD_SDWA(x)                                                                        \
  asm volatile("v_add_u32_sdwa %0, %1, %0 dst_sel:DWORD dst_unused:UNUSED_PAD "             \
               "src0_sel:WORD_1 src1_sel:DWORD" : "+v"(x) : "v"(b));
#define I_XAD(x) asm volatile("v_xad_u32 %0, %1, %2, %0" : "+v"(x) : "v"(b), "v"(c));
#define I_ALIGNBIT(x) asm volatile("v_alignbit_b32 %0, %1, 0, %0" : "+v"(x) : "s"(s));
#define I_BFE(x) asm volatile("v_bfe_i32 %0, %0, 3, 1" : "+v"(x));
#define I_ADD3(x) asm volatile("v_add3_u32 %0, %0, %1, %2" : "+v"(x) : "v"(b), "v"(c));
#define I_LSHL_ADD(x) asm volatile("v_lshl_add_u32 %0, %1, %2, %0" : "+v"(x) : "s"(s), "v"(c));
#define I_PERM(x) asm volatile("v_perm_b32 %0, %0, %1, %2" : "+v"(x) : "v"(b), "v"(c));
#define I_DOT4(x) asm volatile("v_dot4_i32_i8 %0, %1, %2, %0" : "+v"(x) : "v"(b), "v"(c));
#define I_PK_LSHL16(x) asm volatile("v_pk_lshlrev_b16 %0, %1, %0" : "+v"(x) : "v"(c));
#define I_DOT2_U16(x) asm volatile("v_dot2_u32_u16 %0, %1, %2, %0" : "+v"(x) : "v"(b), "v"(c));
#define I_CVT(x) asm volatile("v_cvt_f32_i32_e32 %0, %0" : "+v"(x));
#define I_PK_ASHR16_SGPR(x) asm volatile("v_pk_ashrrev_i16 %0, %0, %1" : "+v"(x) : "s"(s));
#define I_DOT2C_I16(x) asm volatile("v_dot2c_i32_i16 %0, %1, %2" : "+v"(x) : "v"(b), "v"(c));
#define I_DOT2C_I16_SGPR(x) asm volatile("v_dot2c_i32_i16 %0, %1, %2" : "+v"(x) : "s"(s), "v"(c));
#define I_BITOP3(x) asm volatile("v_bitop3_b32 %0, %0, %1, %2 bitop3:0x26" : "+v"(x) : "v"(b), "v"(c));
#define I_BITOP3_SGPR(x) asm volatile("v_bitop3_b32 %0, %0, %1, %2 bitop3:0x26" : "+v"(x) : "s"(s), "v"(c));
#define I_MUL_F32_SGPR(x) asm volatile("v_mul_f32_e32 %0, %1, %0" : "+v"(x) : "s"(s));
#define I_EXP_F32(x) asm volatile("v_exp_f32_e32 %0, %0" : "+v"(x));
#define I_CVT_PKRTZ(x) asm volatile("v_cvt_pkrtz_f16_f32 %0, %0, %1" : "+v"(x) : "v"(b));
#define I_FMA_MIX(x) asm volatile("v_fma_mix_f32 %0, %1, %2, %0 op_sel_hi:[0,1,0]" : "+v"(x) : "v"(b), "v"(c));
#define I_DPP_ROR8(x) asm volatile("v_mov_b32_dpp %0, %0 row_ror:8 row_mask:0xf bank_mask:0xf" : "+v"(x));
// 64-bit shifts: one instruction shifts a register pair (two 32-bit words)
#define I_LSHL64(x) asm volatile("v_lshlrev_b64 %0, %1, %0" : "+v"(x) : "v"(c));
#define I_LSHR64(x) asm volatile("v_lshrrev_b64 %0, %1, %0" : "+v"(x) : "v"(c));
#define KERNEL64(NAME, INS)                                                               \
  __global__ __launch_bounds__(256) void NAME(unsigned* out, unsigned s, unsigned sh) {    \
    unsigned long long a0 = threadIdx.x, a1 = a0 + 1, a2 = a0 + 2, a3 = a0 + 3,           \
                       a4 = a0 + 4, a5 = a0 + 5, a6 = a0 + 6, a7 = a0 + 7;                \
    unsigned c = sh & 3u;                                                                  \
    for (int i = 0; i < N; ++i) {                                                          \
      BODY8(INS)                                                                           \
    }                                                                                      \
    out[blockIdx.x * 256 + threadIdx.x] =                                                  \
        (unsigned)(a0 ^ a1 ^ a2 ^ a3 ^ a4 ^ a5 ^ a6 ^ a7 ^ (a7 >> 32) ^ s);               \
  }

KERNEL(k_add, I_ADD)
KERNEL(k_add_sgpr, I_ADD_SGPR)
KERNEL(k_add_e64, I_ADD_E64)
KERNEL(k_xor, I_XOR)
KERNEL(k_and_lit, I_AND_LIT)
KERNEL(k_mul_f32, I_MUL_F32)
KERNEL(k_fma_f32, I_FMA_F32)
KERNEL(k_lshl, I_LSHL)
KERNEL(k_lshl_sdwa, I_LSHL_SDWA)
KERNEL(k_add_sdwa, I_ADD_SDWA)
KERNEL(k_xad, I_XAD)
KERNEL(k_alignbit, I_ALIGNBIT)
KERNEL(k_bfe, I_BFE)
KERNEL(k_add3, I_ADD3)
KERNEL(k_lshl_add, I_LSHL_ADD)
KERNEL(k_perm, I_PERM)
KERNEL(k_dot4, I_DOT4)
KERNEL(k_pk_lshl16, I_PK_LSHL16)
KERNEL(k_dot2_u16, I_DOT2_U16)
KERNEL(k_cvt, I_CVT)
KERNEL(k_pk_ashr16_sgpr, I_PK_ASHR16_SGPR)
KERNEL(k_dot2c_i16, I_DOT2C_I16)
KERNEL(k_dot2c_i16_sgpr, I_DOT2C_I16_SGPR)
KERNEL(k_bitop3, I_BITOP3)
KERNEL(k_bitop3_sgpr, I_BITOP3_SGPR)
KERNEL(k_mul_f32_sgpr, I_MUL_F32_SGPR)
KERNEL(k_exp_f32, I_EXP_F32)
KERNEL(k_cvt_pkrtz, I_CVT_PKRTZ)
KERNEL(k_fma_mix, I_FMA_MIX)
KERNEL(k_dpp_ror8, I_DPP_ROR8)
KERNEL64(k_lshl64, I_LSHL64)
KERNEL64(k_lshr64, I_LSHR64)

typedef void (*kfn)(unsigned*, unsigned, unsigned);

int main() {
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0) != hipSuccess) return 1;
  const int blocks = cus * 8;  // 8 workgroups of 4 waves per CU: 8 waves per SIMD
  unsigned* out = nullptr;
  if (hipMalloc(&out, (size_t)blocks * 256 * sizeof(unsigned)) != hipSuccess) return 1;
  const struct {
    const char* name;
    kfn f;
  } ks[] = {{"v_add_u32_e32", k_add},        {"v_add_u32_e32 (SGPR src)", k_add_sgpr},
            {"v_add_u32_e64", k_add_e64},    {"v_xor_b32_e32", k_xor},
            {"v_and_b32_e32 (literal)", k_and_lit}, {"v_mul_f32_e32", k_mul_f32},
            {"v_fma_f32", k_fma_f32},        {"v_lshlrev_b32_e32", k_lshl},
            {"v_lshlrev_b32_sdwa (SGPR)", k_lshl_sdwa}, {"v_add_u32_sdwa", k_add_sdwa},
            {"v_xad_u32", k_xad},            {"v_alignbit_b32 (SGPR)", k_alignbit},
            {"v_bfe_i32", k_bfe},            {"v_add3_u32", k_add3},
            {"v_lshl_add_u32 (SGPR)", k_lshl_add}, {"v_perm_b32", k_perm},
            {"v_dot4_i32_i8", k_dot4},       {"v_pk_lshlrev_b16", k_pk_lshl16},
            {"v_dot2_u32_u16", k_dot2_u16},  {"v_cvt_f32_i32_e32", k_cvt},
            {"v_pk_ashrrev_i16 (SGPR)", k_pk_ashr16_sgpr}, {"v_dot2c_i32_i16", k_dot2c_i16},
            {"v_dot2c_i32_i16 (SGPR)", k_dot2c_i16_sgpr}, {"v_bitop3_b32", k_bitop3},
            {"v_bitop3_b32 (SGPR)", k_bitop3_sgpr}, {"v_mul_f32_e32 (SGPR)", k_mul_f32_sgpr},
            {"v_exp_f32_e32", k_exp_f32},    {"v_cvt_pkrtz_f16_f32", k_cvt_pkrtz},
            {"v_fma_mix_f32", k_fma_mix},    {"v_mov_b32_dpp row_ror:8", k_dpp_ror8},
            {"v_lshlrev_b64", k_lshl64},     {"v_lshrrev_b64", k_lshr64}};
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return 1;
  printf("%d CUs; wave64 instructions per ns per CU (2.4 = one per cycle per CU at 2.4 GHz)\n", cus);
  for (const auto& k : ks) {
    float ms = 0.0f;
    for (int rep = 0; rep < 3; ++rep) {  // the last of three launches is reported
      if (hipEventRecord(e0) != hipSuccess) return 1;
      hipLaunchKernelGGL(k.f, dim3(blocks), dim3(256), 0, 0, out, 0x12345u, 0x0505u);
      if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) return 1;
      if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) return 1;
    }
    const double insts = (double)blocks * 4 * N * 8;
    printf("%-28s %7.3f ms %7.3f\n", k.name, ms, insts / (ms * 1e6) / cus);
  }
  if (hipFree(out) != hipSuccess) return 1;
  return 0;
}
