// pot_decode_attention_noalloc: pot_decode_attention on a workspace the
// library owns, for callers that cannot allocate device memory (code under
// HIP graph capture, tight serving loops).
//
// The workspace (prepared query operands and key-split partials) lives in a
// static device array of POT_NOALLOC_SCRATCH_BYTES, one copy per GPU, held
// from the library's load until the process ends. Host code never uses the
// array's name as an address (in host code it names a host-side stand-in):
// the device address of the current GPU's copy is looked up once per device
// with hipGetSymbolAddress and cached, and only that address is handed to the
// kernels, exactly as a caller's workspace would be. The decode kernels write
// every workspace word they read, so nothing needs clearing between calls.
// Every call on one GPU shares that GPU's copy: calls that overlap in time on
// one GPU (two streams, or two host threads) race on it.
#include <hip/hip_runtime.h>

#include <atomic>

#include "pot_attn.h"
#include "pot_launch.hpp"

namespace potattn {
namespace {

constexpr size_t kScratchBytes = POT_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of the current GPU's scratch copy (looked up once per
// device, with that device current).
hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return hipSuccess;
}

}  // namespace
}  // namespace potattn

extern "C" pot_status pot_decode_attention_noalloc(
    const pot_format* fmt, const float* q, const uint8_t* codes_se, const uint8_t* codes_m,
    const float* key_scale, const uint16_t* v_cache, int64_t t_cap,
    const int32_t* kv_head_of_q, int32_t B, int32_t Hq, int32_t Hkv, int32_t T, float* out,
    pot_debug* dbg, void* stream) {
  using namespace potattn;
  // the shape's workspace bound, checked on the host before any HIP call
  const int force = dbg ? dbg->force_splits : 0;
  const size_t need = force > 0 ? pot_decode_workspace_bytes_for_splits(B, Hq, Hkv, T, force)
                                 : pot_decode_workspace_bytes(B, Hq, Hkv, T);
  if (need > kScratchBytes)
    return report_error(POT_ERR_WORKSPACE,
                        "pot_decode_attention_noalloc: this shape needs %zu bytes of "
                        "workspace; the static scratch holds %zu (split the batch, or use "
                        "pot_decode_attention with a caller workspace)",
                        need, kScratchBytes);
  void* ws = nullptr;
  const hipError_t e = scratch_address(&ws);
  if (e != hipSuccess)
    return report_error(POT_ERR_HIP, "pot_decode_attention_noalloc: scratch address: %s",
                        hipGetErrorString(e));
  return pot_decode_attention(fmt, q, codes_se, codes_m, key_scale, v_cache, t_cap,
                              kv_head_of_q, B, Hq, Hkv, T, out, ws, kScratchBytes, dbg, stream);
}
