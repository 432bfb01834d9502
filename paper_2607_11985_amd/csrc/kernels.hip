// kernels.hip -- precompiled gfx950 kernels: the schedule interpreter for every
// circuit (resident and streaming), the reductions of the streaming path, the
// loss cotangent, and the launchers.  The device code lives in vqc_device.h.
#include <hip/hip_runtime.h>

#include <mutex>

#include "vqc.h"
#include "vqc_device.h"
#include "vqc_internal.h"

// The workspace of vqc_train_step_noalloc: a static device array, one copy per
// GPU that loads this library, held until the process ends.  In host code this
// name is only a stand-in for the registration of the variable: kernels receive
// the device address that scratch_pointer() looks up once per device.
static __device__ __align__(256) unsigned char scratch[VQC_NOALLOC_SCRATCH_BYTES];

namespace vqc {
namespace {

template <int WG, bool BWD, int R>
__global__ void __launch_bounds__(WG) resident_kernel(const TileArgs A) {
  extern __shared__ __align__(16) unsigned char smem[];
  resident_body<WG, BWD, R, InterpSched>(A, smem);
}

template <int WG, int R>
__global__ void __launch_bounds__(WG) resident_step_kernel(const TileArgs A) {
  extern __shared__ __align__(16) unsigned char smem[];
  resident_step_body<WG, R, InterpSched, InterpSched>(A, smem);
}

template <bool BWD, int R>
__global__ void __launch_bounds__(1 << (kMaxTileQubits - R)) stream_kernel(const PassArgs A) {
  extern __shared__ __align__(16) unsigned char smem[];
  stream_body<BWD, R, kMaxTileQubits, InterpSched>(A, smem);
}

__global__ void reduce_e_kernel(int64_t B, int ng, int n, const float* __restrict__ epart,
                                float* __restrict__ e) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * n) return;
  const int64_t b = i / n;
  const int q = (int)(i - b * n);
  float v = 0.f;
#pragma unroll 8  // loads in flight together; the sum keeps its order
  for (int g = 0; g < (1 << ng); ++g) v += epart[((b << ng) + g) * n + q];
  e[i] = v;
}

// The streaming training step's <Z> rows from the tiles' partials, then the
// loss head's cotangent rows, in one launch: a block holds whole rows (256 / n
// samples), which it passes to the loss head through LDS.
__global__ void __launch_bounds__(256) reduce_e_loss_kernel(int64_t B, int ng, int n,
                                                            const float* __restrict__ epart,
                                                            float* __restrict__ e, int kind,
                                                            int64_t norm,
                                                            const float* __restrict__ y,
                                                            float* __restrict__ g) {
  __shared__ float rows[256];
  const int spb = 256 / n;
  const int t = threadIdx.x;
  const int ls = t / n, q = t - ls * n;
  const int64_t b = (int64_t)blockIdx.x * spb + ls;
  const bool on = ls < spb && b < B;
  if (on) {
    float v = 0.f;
#pragma unroll 8  // loads in flight together; the sum keeps its order
    for (int gi = 0; gi < (1 << ng); ++gi) v += epart[((b << ng) + gi) * n + q];
    e[b * n + q] = v;
    rows[t] = v;
  }
  __syncthreads();
  if (on) g[b * n + q] = loss_cot(kind, rows + ls * n, y ? y[b] : 0.f, n, q, norm);
}

__global__ void reduce_grad_kernel(int64_t B, int ng, int n_slots, int P, int F,
                                   const float* __restrict__ gpart, float* __restrict__ dparams,
                                   float* __restrict__ dinputs) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * n_slots) return;
  const int64_t b = i / n_slots;
  const int s = (int)(i - b * n_slots);
  float v = 0.f;
#pragma unroll 8  // loads in flight together; the sum keeps its order
  for (int g = 0; g < (1 << ng); ++g) v += gpart[((b << ng) + g) * n_slots + s];
  if (s < P) {
    if (dparams) dparams[b * P + s] = v;
  } else if (dinputs) {
    dinputs[b * F + (s - P)] = v;
  }
}

// One workgroup per column: thread t adds rows t, t + 256, ... in order, then a
// fixed tree over the threads.  Deterministic for a given batch size.
__global__ void __launch_bounds__(256) sum_rows_kernel(int64_t B, int P,
                                                       const float* __restrict__ rows,
                                                       float* __restrict__ out) {
  __shared__ float part[256];
  const int p = blockIdx.x;
  float v = 0.f;
  for (int64_t b = threadIdx.x; b < B; b += 256) v += rows[b * P + p];
  part[threadIdx.x] = v;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) part[threadIdx.x] += part[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[p] = part[0];
}

// Central differences: d L / d slot s of row b = sum_q g[b,q] (E(+h) - E(-h)) / 2h,
// with the shifted copies laid out as the forward's fd_slots mode writes them.
__global__ void fd_combine_kernel(int64_t B, int NS, int base, int P, int F, int n, float h,
                                  const float* __restrict__ ev, const float* __restrict__ g,
                                  float* __restrict__ dparams, float* __restrict__ dinputs) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * NS) return;
  const int64_t b = i / NS;
  const int s = (int)(i - b * NS);
  const float* ep = ev + ((b * NS + s) * 2) * n;
  const float* em = ep + n;
  const float* gb = g + b * n;
  float v = 0.f;
  for (int q = 0; q < n; ++q) v += gb[q] * (ep[q] - em[q]);
  v /= 2.f * h;
  const int slot = base + s;
  if (slot < P) {
    if (dparams) dparams[b * P + slot] = v;
  } else if (dinputs) {
    dinputs[b * F + (slot - P)] = v;
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0.f;
}

// rows b < B of a batch of `norm` samples (the MSE losses average over norm)
__global__ void loss_grad_kernel(int kind, int64_t B, int64_t norm, int n,
                                 const float* __restrict__ e, const float* __restrict__ y,
                                 float* __restrict__ g) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const float* eb = e + b * n;
  float* gb = g + b * n;
  const float yb = y ? y[b] : 0.f;
  for (int j = 0; j < n; ++j) gb[j] = loss_cot(kind, eb, yb, n, j, norm);
}

// ------------------------------------------------------------ launchers

// Resident instantiations: R in {2, 3, 4}, workgroups of 64..1024 threads.
template <typename F>
int by_wg(int wg, F&& f) {
  switch (wg) {
    case 64: return f(IC<64>{});
    case 128: return f(IC<128>{});
    case 256: return f(IC<256>{});
    case 512: return f(IC<512>{});
    case 1024: return f(IC<1024>{});
    default: return (int)hipErrorInvalidValue;
  }
}

template <typename F>
int by_res_r(int r, F&& f) {
  switch (r) {
    case 2: return f(IC<2>{});
    case 3: return f(IC<3>{});
    case 4: return f(IC<4>{});
    default: return (int)hipErrorInvalidValue;
  }
}

template <bool BWD>
int launch_resident(const Plan& p, const TileArgs& a, int64_t blocks, void* stream) {
  const size_t lds = BWD ? p.lds_bwd : p.lds_fwd;
  return by_res_r(p.R, [&](auto Rc) {
    constexpr int R = decltype(Rc)::value;
    return by_wg(p.WG, [&](auto Wc) {
      constexpr int WG = decltype(Wc)::value;
      hipLaunchKernelGGL((resident_kernel<WG, BWD, R>), dim3((unsigned)blocks), dim3(WG), lds,
                         (hipStream_t)stream, a);
      return (int)hipGetLastError();
    });
  });
}

unsigned grid_1d(int64_t count, int threads) { return (unsigned)((count + threads - 1) / threads); }

int set_attr(const void* f, size_t lds) {
  return (int)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

}  // namespace

int prepare_kernels(const Plan& p) {
  if (p.path == VQC_PATH_STREAM) {
    int e = p.Rf == 5 ? set_attr((const void*)stream_kernel<false, 5>, p.lds_fwd)
                      : set_attr((const void*)stream_kernel<false, 4>, p.lds_fwd);
    if (e) return e;
    return p.Rb == 5 ? set_attr((const void*)stream_kernel<true, 5>, p.lds_bwd)
                     : set_attr((const void*)stream_kernel<true, 4>, p.lds_bwd);
  }
  return by_res_r(p.R, [&](auto Rc) {
    constexpr int R = decltype(Rc)::value;
    return by_wg(p.WG, [&](auto Wc) {
      constexpr int WG = decltype(Wc)::value;
      int e = set_attr((const void*)resident_kernel<WG, false, R>, p.lds_fwd);
      if (e) return e;
      e = set_attr((const void*)resident_step_kernel<WG, R>, p.lds_step);
      if (e) return e;
      return set_attr((const void*)resident_kernel<WG, true, R>, p.lds_bwd);
    });
  });
}

int launch_resident_forward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream) {
  return launch_resident<false>(plan, a, blocks, stream);
}

int launch_resident_backward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream) {
  return launch_resident<true>(plan, a, blocks, stream);
}

int launch_resident_step(const Plan& p, const TileArgs& a, int64_t blocks, void* stream) {
  return by_res_r(p.R, [&](auto Rc) {
    constexpr int R = decltype(Rc)::value;
    return by_wg(p.WG, [&](auto Wc) {
      constexpr int WG = decltype(Wc)::value;
      hipLaunchKernelGGL((resident_step_kernel<WG, R>), dim3((unsigned)blocks), dim3(WG),
                         p.lds_step, (hipStream_t)stream, a);
      return (int)hipGetLastError();
    });
  });
}

int launch_stream_pass(const Plan& p, bool bwd, const PassArgs& a, int64_t blocks,
                       void* stream) {
  const int R = bwd ? p.Rb : p.Rf;
  const size_t lds = bwd ? p.lds_bwd : p.lds_fwd;
  const dim3 grid((unsigned)blocks);
  if (bwd && R == 5)
    hipLaunchKernelGGL((stream_kernel<true, 5>), grid, dim3(1 << 9), lds, (hipStream_t)stream, a);
  else if (bwd)
    hipLaunchKernelGGL((stream_kernel<true, 4>), grid, dim3(1 << 10), lds, (hipStream_t)stream, a);
  else if (R == 5)
    hipLaunchKernelGGL((stream_kernel<false, 5>), grid, dim3(1 << 9), lds, (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL((stream_kernel<false, 4>), grid, dim3(1 << 10), lds, (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

int launch_reduce_e(int64_t batch, int ng, int n, const float* epart, float* e, void* stream) {
  hipLaunchKernelGGL(reduce_e_kernel, dim3(grid_1d(batch * n, 256)), dim3(256), 0,
                     (hipStream_t)stream, batch, ng, n, epart, e);
  return (int)hipGetLastError();
}

int launch_reduce_e_loss(int64_t batch, int ng, int n, const float* epart, float* e, int kind,
                         int64_t norm, const float* y, float* g, void* stream) {
  const int spb = 256 / n;
  hipLaunchKernelGGL(reduce_e_loss_kernel, dim3((unsigned)((batch + spb - 1) / spb)), dim3(256), 0,
                     (hipStream_t)stream, batch, ng, n, epart, e, kind, norm, y, g);
  return (int)hipGetLastError();
}

int launch_reduce_grad(int64_t batch, int ng, int n_slots, int P, int F, const float* gpart,
                       float* dparams, float* dinputs, void* stream) {
  if (batch * n_slots == 0) return 0;
  hipLaunchKernelGGL(reduce_grad_kernel, dim3(grid_1d(batch * n_slots, 256)), dim3(256), 0,
                     (hipStream_t)stream, batch, ng, n_slots, P, F, gpart, dparams, dinputs);
  return (int)hipGetLastError();
}

int launch_sum_rows(int64_t batch, int P, const float* rows, float* out, void* stream) {
  if (P == 0) return 0;
  hipLaunchKernelGGL(sum_rows_kernel, dim3((unsigned)P), dim3(256), 0, (hipStream_t)stream, batch,
                     P, rows, out);
  return (int)hipGetLastError();
}

int launch_fd_combine(int64_t batch, int NS, int base, int P, int F, int n, float h,
                      const float* ev, const float* g, float* dparams, float* dinputs,
                      void* stream) {
  if (batch * NS == 0) return 0;
  hipLaunchKernelGGL(fd_combine_kernel, dim3(grid_1d(batch * NS, 256)), dim3(256), 0,
                     (hipStream_t)stream, batch, NS, base, P, F, n, h, ev, g, dparams, dinputs);
  return (int)hipGetLastError();
}

int launch_fill_zero(float* p, int64_t count, void* stream) {
  if (count == 0) return 0;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_1d(count, 256)), dim3(256), 0,
                     (hipStream_t)stream, p, count);
  return (int)hipGetLastError();
}

int scratch_pointer(int device, void** out) {
  static std::mutex mu;
  static void* ptr[kScratchDevices] = {};
  *out = nullptr;
  if (device < 0 || device >= kScratchDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return (int)e;
    if (cur != device) return (int)hipErrorInvalidDevice;  // the caller makes it current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    if (!p) return (int)hipErrorInvalidSymbol;
    ptr[device] = p;
  }
  *out = ptr[device];
  return 0;
}

int launch_loss_grad(int kind, int64_t batch, int64_t norm, int n, const float* e,
                     const float* y, float* g, void* stream) {
  const int threads = 256;
  const int64_t blocks = (batch + threads - 1) / threads;
  hipLaunchKernelGGL(loss_grad_kernel, dim3((unsigned)blocks), dim3(threads), 0,
                     (hipStream_t)stream, kind, batch, norm, n, e, y, g);
  return (int)hipGetLastError();
}

}  // namespace vqc
