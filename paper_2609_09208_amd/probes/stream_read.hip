// Achievable HBM read bandwidth on this device: every lane streams 16-byte
// loads over a buffer far larger than the last-level cache and folds them into
// a register; one word per workgroup is written at the end. The grid is a few
// workgroups per CU with a grid-stride loop, the same access shape as the
// decode kernels' code and value streams (one 16-byte load per lane). Each
// grid is run with plain loads and with non-temporal loads (the nt hint the
// decode kernels put on their streams).
//
// Build and run on a gfx950 device:
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//         -o stream_read paper_2609_09208_amd/probes/stream_read.hip && ./stream_read
#include <hip/hip_runtime.h>

#include <cstdio>

typedef unsigned u32x4v __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ uint4 ld(const uint4* p) {
  if constexpr (NT) {
    const u32x4v v = __builtin_nontemporal_load(reinterpret_cast<const u32x4v*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
  } else {
    return *p;
  }
}

template <bool NT>
__global__ __launch_bounds__(256) void read_kernel(const uint4* __restrict__ src, size_t n16,
                                                   unsigned* __restrict__ out) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  unsigned acc = 0;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  // four independent loads in flight per lane per iteration
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = ld<NT>(src + i), b = ld<NT>(src + i + stride), c = ld<NT>(src + i + 2 * stride),
                d = ld<NT>(src + i + 3 * stride);
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^
           d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const uint4 a = ld<NT>(src + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  __shared__ unsigned red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned r = 0;
    for (int k = 0; k < 256; ++k) r ^= red[k];
    out[blockIdx.x] = r;
  }
}

int main() {
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0) != hipSuccess) return 1;
  const size_t bytes = (size_t)4 << 30;  // 4 GiB, 16x the last-level cache
  const size_t n16 = bytes / 16;
  uint4* src = nullptr;
  unsigned* out = nullptr;
  if (hipMalloc(&src, bytes) != hipSuccess) return 1;
  if (hipMemset(src, 1, bytes) != hipSuccess) return 1;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return 1;
  printf("%d CUs, %zu MiB read per launch\n", cus, bytes >> 20);
  for (int nt = 0; nt < 2; ++nt)
  for (int per_cu : {2, 4, 8, 16}) {
    const int blocks = cus * per_cu;
    if (hipMalloc(&out, (size_t)blocks * sizeof(unsigned)) != hipSuccess) return 1;
    float best = 1e30f, sum = 0.0f;
    const int reps = 10;
    for (int r = 0; r < reps + 2; ++r) {
      if (hipEventRecord(e0) != hipSuccess) return 1;
      if (nt)
        hipLaunchKernelGGL(read_kernel<true>, dim3(blocks), dim3(256), 0, 0, src, n16, out);
      else
        hipLaunchKernelGGL(read_kernel<false>, dim3(blocks), dim3(256), 0, 0, src, n16, out);
      if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) return 1;
      float ms = 0.0f;
      if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) return 1;
      if (r >= 2) {
        sum += ms;
        best = ms < best ? ms : best;
      }
    }
    printf("%s loads, workgroups/CU %2d: mean %.3f ms = %.0f GB/s, best %.3f ms = %.0f GB/s\n",
           nt ? "nt   " : "plain", per_cu, sum / reps, bytes / (sum / reps * 1e-3) / 1e9, best,
           bytes / (best * 1e-3) / 1e9);
    if (hipFree(out) != hipSuccess) return 1;
  }
  if (hipFree(src) != hipSuccess) return 1;
  return 0;
}
