// probes.hip -- peak microbenchmarks for the roofline fractions (built into
// libvqc_probes.so, separate from the engine; bench.py --probe runs them).
//
//   fma : eight independent fp32 FMA chains per thread, compiled with the
//         engine's flags (packed FP32 off): the VALU issue ceiling the engine's
//         kernels can reach.  2 flops per FMA.
//   lds128 / lds32 : every thread reads LDS with 16-byte / 4-byte loads at
//         consecutive addresses per lane (no bank conflicts), one add per
//         loaded float; bytes = loads x width.
// Each kernel writes one value per thread so that nothing is optimised away.
// Grids are sized on the host from the arguments; every access is in bounds.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kThreads = 256;
constexpr int kChains = 8;
constexpr int kUnroll = 16;
constexpr int kLdsFloat4 = 4096;  // 64 KiB of LDS per workgroup

__global__ void __launch_bounds__(kThreads) fma_probe(float* __restrict__ out, int iters, float a,
                                                      float b) {
  const int gid = blockIdx.x * kThreads + threadIdx.x;
  float x[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) x[c] = (float)(threadIdx.x + c) * 1e-3f;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int c = 0; c < kChains; ++c) x[c] = __builtin_fmaf(x[c], a, b);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += x[c];
  out[gid] = s;
}

__global__ void __launch_bounds__(kThreads) lds128_probe(float* __restrict__ out, int iters) {
  __shared__ float4 buf[kLdsFloat4];
  const int t = threadIdx.x;
  for (int i = t; i < kLdsFloat4; i += kThreads)
    buf[i] = make_float4((float)i, (float)(i + 1), (float)(i + 2), (float)(i + 3));
  __syncthreads();
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float4 v = buf[(t + (i * 8 + u) * kThreads) & (kLdsFloat4 - 1)];
      acc.x += v.x;
      acc.y += v.y;
      acc.z += v.z;
      acc.w += v.w;
    }
  }
  out[blockIdx.x * kThreads + t] = acc.x + acc.y + acc.z + acc.w;
}

__global__ void __launch_bounds__(kThreads) lds32_probe(float* __restrict__ out, int iters) {
  __shared__ float buf[4 * kLdsFloat4];
  const int t = threadIdx.x;
  for (int i = t; i < 4 * kLdsFloat4; i += kThreads) buf[i] = (float)i;
  __syncthreads();
  float acc0 = 0.f, acc1 = 0.f;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < 8; u += 2) {
      acc0 += buf[(t + (i * 8 + u) * kThreads) & (4 * kLdsFloat4 - 1)];
      acc1 += buf[(t + (i * 8 + u + 1) * kThreads) & (4 * kLdsFloat4 - 1)];
    }
  }
  out[blockIdx.x * kThreads + t] = acc0 + acc1;
}

}  // namespace

extern "C" {

// out: device array of blocks * 256 floats.  Returns a hipError_t value.
int vqc_probe_fma(float* out, int blocks, int iters, void* stream) {
  hipLaunchKernelGGL(fma_probe, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream, out, iters,
                     0.999f, 1e-3f);
  return (int)hipGetLastError();
}

int vqc_probe_lds(float* out, int blocks, int iters, int width, void* stream) {
  if (width == 16)
    hipLaunchKernelGGL(lds128_probe, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream, out,
                       iters);
  else
    hipLaunchKernelGGL(lds32_probe, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream, out,
                       iters);
  return (int)hipGetLastError();
}

// flops (fma) or LDS bytes (lds) one launch performs
double vqc_probe_work(int kind, int blocks, int iters, int width) {
  const double threads = (double)blocks * kThreads;
  if (kind == 0) return threads * iters * kUnroll * kChains * 2.0;
  return threads * iters * 8.0 * width;
}

}  // extern "C"
