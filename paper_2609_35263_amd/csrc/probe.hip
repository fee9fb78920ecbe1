// Matrix-core rate and shader-clock probe (a measurement tool beside the attention path).
#include <hip/hip_runtime.h>

#include "wavepp_probe.h"
#include "internal.h"

namespace wavepp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kProbeThreads = 512;

__device__ __forceinline__ uint32_t mix32(uint32_t x) {   // an integer hash (xorshift-multiply)
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(int iters, int random_operands,
                                                                   float* __restrict__ sink,
                                                                   unsigned long long* __restrict__ clocks) {
  const int tid = threadIdx.x;
  // operands from the thread index, so that nothing folds at compile time: a few small values, or
  // N(0,1)-like bf16 values with random mantissa bits (as attention operands have)
  bf16x8 a, b;
  const uint32_t seed = (blockIdx.x * kProbeThreads + tid) * 16u;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (random_operands) {
      const uint32_t ha = mix32(seed + e), hb = mix32(seed + 8 + e);
      a[e] = static_cast<__bf16>((float(ha & 0xffffu) - 32768.0f) * (1.0f / 16384.0f));
      b[e] = static_cast<__bf16>((float(hb & 0xffffu) - 32768.0f) * (1.0f / 16384.0f));
    } else {
      a[e] = static_cast<__bf16>(float((tid + e) & 7) * 0.125f);
      b[e] = static_cast<__bf16>(float((tid * 3 + e) & 7) * 0.0625f);
    }
  }
  f32x16 acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f32x16{};
  const bool rec = blockIdx.x == 0 && tid == 0;
  unsigned long long t0 = 0, r0 = 0;
  if (rec) {
    t0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  if (rec) {
    const unsigned long long t1 = __builtin_amdgcn_s_memtime();
    const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
    clocks[0] = t0;
    clocks[1] = r0;
    clocks[2] = t1;
    clocks[3] = r1;
  }
  sink[int64_t(blockIdx.x) * kProbeThreads + tid] = s;
}


// Read-only HBM stream: every thread reads 16 bytes from each of four 4 KiB-apart positions per
// round (grid-stride), folds them with XOR and writes one word, so the bytes read are exactly the
// buffer once and nothing is written back but the per-thread words.
constexpr int kReadThreads = 256;
typedef uint32_t u32x4p __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kReadThreads) void hbm_read_probe_kernel(const u32x4p* __restrict__ src, int64_t n16,
                                                                      uint32_t* __restrict__ sink) {
  u32x4p acc = {0u, 0u, 0u, 0u};
  const int64_t stride = int64_t(gridDim.x) * kReadThreads * 4;
  for (int64_t i = int64_t(blockIdx.x) * kReadThreads * 4 + threadIdx.x; i < n16; i += stride) {
    const u32x4p a = src[i];
    const u32x4p b = (i + kReadThreads < n16) ? src[i + kReadThreads] : u32x4p{0u, 0u, 0u, 0u};
    const u32x4p c = (i + 2 * kReadThreads < n16) ? src[i + 2 * kReadThreads] : u32x4p{0u, 0u, 0u, 0u};
    const u32x4p d = (i + 3 * kReadThreads < n16) ? src[i + 3 * kReadThreads] : u32x4p{0u, 0u, 0u, 0u};
    acc ^= a ^ b ^ c ^ d;
  }
  sink[int64_t(blockIdx.x) * kReadThreads + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}
}  // namespace
}  // namespace wavepp

extern "C" int wavepp_probe_mfma(int32_t workgroups, int32_t iters, int32_t random_operands, float* sink,
                                 unsigned long long* clocks, hipStream_t stream) {
  using namespace wavepp;
  clear_error();
  if (workgroups <= 0 || iters <= 0) return set_error(WAVEPP_EINVAL, "workgroups and iters must be positive");
  if (!sink || !clocks) return set_error(WAVEPP_EINVAL, "sink / clocks is NULL");
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(workgroups), dim3(kProbeThreads), 0, stream, iters,
                     random_operands ? 1 : 0, sink, clocks);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_hip_error(e, "probe launch");
  return WAVEPP_OK;
}

extern "C" int wavepp_probe_hbm_read(const void* src, int64_t bytes, int32_t workgroups, uint32_t* sink,
                                     hipStream_t stream) {
  using namespace wavepp;
  clear_error();
  if (workgroups <= 0 || bytes <= 0) return set_error(WAVEPP_EINVAL, "workgroups and bytes must be positive");
  if (bytes % 16 != 0) return set_error(WAVEPP_EINVAL, "bytes must be a multiple of 16");
  if (!src || !sink) return set_error(WAVEPP_EINVAL, "src / sink is NULL");
  if (reinterpret_cast<uintptr_t>(src) % 16 != 0) return set_error(WAVEPP_EINVAL, "src must be 16-byte aligned");
  hipLaunchKernelGGL(hbm_read_probe_kernel, dim3(workgroups), dim3(kReadThreads), 0, stream,
                     static_cast<const u32x4p*>(src), bytes / 16, sink);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_hip_error(e, "probe launch");
  return WAVEPP_OK;
}
