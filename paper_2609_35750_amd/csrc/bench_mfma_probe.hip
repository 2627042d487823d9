// Benchmark-only probe (libkvs_bench.so, loaded by bench.py; not part of the
// libkvs ABI): the dense bf16 matrix-core rate the device sustains on
// changing data, to report kernel efficiency against a measured peak beside
// the published one.
//
// Every wave runs eight independent accumulation chains of
// v_mfma_f32_32x32x16_bf16, each chain with its own operands drawn from a
// per-lane hash (bf16 values of magnitude 0.5 - 2 with random sign and
// mantissa), so consecutive products feed the matrix core different bits, as
// the attention kernels do: on constant operands the shader clock runs
// higher than on real data, which would overstate the attainable rate.
//
//   extern "C" int kvs_bench_mfma_rate(double* tflops, void* stream)
//   Synchronous; four 256-thread workgroups per compute unit, timed with HIP
//   events on `stream` after one warm-up launch.  Returns 0, 1 for a NULL
//   tflops, or the hipError_t of a failed call.
#include <hip/hip_runtime.h>
#include <stdint.h>

// Target of the never-taken store that keeps the products live (external
// linkage: a store to a variable nothing in this file reads would be dropped).
__device__ float kvs_bench_probe_sink;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint32_t mix(uint32_t x) {   // 32-bit integer hash (xorshift-multiply)
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

__device__ __forceinline__ bf16x8 random_operand(uint32_t seed) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t h = mix(seed * 8u + (uint32_t)e);
    // sign | exponent 126 or 127 (0.5 .. 2) | 7 random mantissa bits
    const uint16_t bits = (uint16_t)(((h >> 31) << 15) | ((126u + ((h >> 7) & 1u)) << 7) | (h & 0x7fu));
    r[e] = __builtin_bit_cast(__bf16, bits);
  }
  return r;
}

__global__ void __launch_bounds__(256) mfma_probe_kernel(int iters) {
  const uint32_t lane = blockIdx.x * 256u + threadIdx.x;
  bf16x8 a[8], b[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    a[k] = random_operand(lane * 16u + (uint32_t)k);
    b[k] = random_operand(lane * 16u + 8u + (uint32_t)k);
  }
  f32x16 c[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) c[k] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[k], b[k], c[k], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c[k][r];
  if (s == 1.234567e30f) kvs_bench_probe_sink = s;   // never true in practice
}

}  // namespace

extern "C" int kvs_bench_mfma_rate(double* tflops, void* stream_) {
  if (!tflops) return 1;
  hipStream_t stream = (hipStream_t)stream_;
  int dev = 0, ncu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return (int)e;
  const int blocks = 4 * ncu, iters = 4096;
  hipEvent_t t0, t1;
  if ((e = hipEventCreate(&t0)) != hipSuccess) return (int)e;
  if ((e = hipEventCreate(&t1)) != hipSuccess) {
    (void)hipEventDestroy(t0);
    return (int)e;
  }
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(256), 0, stream, iters);   // warm-up
  (void)hipEventRecord(t0, stream);
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(256), 0, stream, iters);
  (void)hipEventRecord(t1, stream);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipEventSynchronize(t1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, t0, t1);
  (void)hipEventDestroy(t0);
  (void)hipEventDestroy(t1);
  if (e != hipSuccess) return (int)e;
  const double flops = (double)blocks * 4 * iters * 8 * (32.0 * 32 * 16 * 2);
  *tflops = ms > 0.f ? flops / (ms * 1e-3) / 1e12 : 0.0;
  return 0;
}
