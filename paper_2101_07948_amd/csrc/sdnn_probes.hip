// Measurement probes (see include/sdnn_probes.h): the FMA issue rate and the LDS read
// rate of 1 KB rows that the panel kernel's inner loop depends on.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sdnn_probes.h"

namespace {

constexpr int kBlocks = 256, kThreads = 1024;  // one 16-wave workgroup per CU

// 8 independent FMA chains per thread, each step 2 FMAs (x*a + b, then y*a + c) so
// that no chain can be folded; unpacked because the build disables packed FP32.
__global__ __launch_bounds__(kThreads) void fma_probe(int iters, float* out) {
  const float a = 1.0f + 1e-7f * (float)(threadIdx.x & 7), b = 1e-7f, c = -1e-7f;
  float x[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] = (float)(threadIdx.x + k);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      x[k] = fmaf(x[k], a, b);
      x[k] = fmaf(x[k], a, c);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += x[k];
  out[blockIdx.x * kThreads + threadIdx.x] = s;
}

// 128 KB of LDS; each wave reads 8 pseudo-random 1 KB rows per iteration, lane l the
// bytes 16l..16l+15 of each row (the panel kernel's access pattern).
__global__ __launch_bounds__(kThreads) void lds_probe(int iters, float* out) {
  __shared__ __attribute__((aligned(16))) float lds[32768];
  for (int i = threadIdx.x; i < 32768; i += kThreads) lds[i] = (float)(i & 7);
  __syncthreads();
  const uint32_t lane16 = (threadIdx.x & 63) * 16;
  uint32_t r = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) * 2654435761u + 12345u;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int it = 0; it < iters; ++it) {
    float4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      r = r * 1664525u + 1013904223u;  // wave-uniform row in 0..127
      v[j] = *(const float4*)((const char*)lds + (((r >> 25) << 10) | lane16));
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      acc.x += v[j].x; acc.y += v[j].y; acc.z += v[j].z; acc.w += v[j].w;
    }
  }
  out[blockIdx.x * kThreads + threadIdx.x] = acc.x + acc.y + acc.z + acc.w;
}

}  // namespace

extern "C" {

int64_t sdnn_probe_out_floats(void) { return (int64_t)kBlocks * kThreads; }

int32_t sdnn_probe_fma(int32_t iters, float* out, void* stream) {
  if (iters < 0 || !out) return (int32_t)hipErrorInvalidValue;
  hipLaunchKernelGGL(fma_probe, dim3(kBlocks), dim3(kThreads), 0, (hipStream_t)stream, iters, out);
  return (int32_t)hipGetLastError();
}

int32_t sdnn_probe_lds_read(int32_t iters, float* out, void* stream) {
  if (iters < 0 || !out) return (int32_t)hipErrorInvalidValue;
  hipLaunchKernelGGL(lds_probe, dim3(kBlocks), dim3(kThreads), 0, (hipStream_t)stream, iters, out);
  return (int32_t)hipGetLastError();
}

}  // extern "C"
