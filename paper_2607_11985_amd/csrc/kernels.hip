// kernels.hip -- gfx950 kernels of the batched VQC engine.
//
// Resident path (n <= 14): one launch runs the whole circuit for a tile of
// samples (Algorithm 1, execute phase):
//   1. per-sample angle table: (cos, sin)(theta/2) for every rotation
//      occurrence, theta read from params / inputs, constants from the
//      compiled schedule (parameter resolution);
//   2. state init |0...0> in registers (16 amplitudes per thread);
//   3. the instruction stream: register-bit rotations and CNOTs (VALU only),
//      diagonal RZ / CZ on any bit, LDS exchanges that move other qubits onto
//      the register bits;
//   4. epilogue: <Z_j> reduction (Algorithm 1, return statement) and, when
//      training, the final state saved for the adjoint sweep.
// The adjoint kernel reloads psi_G, forms lambda = (sum_j g_j Z_j) psi_G and
// walks the schedule backwards: for every rotation R_P(t) it accumulates
// dL/dt = Im <lambda| P |psi> and then un-applies the gate on both states
// (psi <- U^dagger psi, lambda <- U^dagger lambda).  This is the exact gradient
// of Sec. 3 "Gate Application and Differentiation" with O(state) memory.
#include <hip/hip_runtime.h>

#include "vqc.h"
#include "vqc_internal.h"

namespace vqc {
namespace {

// A thread's 16 amplitudes as plain scalars (real and imaginary parts kept in
// separate arrays so every access has a constant index and stays in VGPRs).
struct St {
  float r[kRegAmps];
  float i[kRegAmps];
};

// ------------------------------------------------------------------ gates
// R_P(t) = exp(-i t P / 2) with c = cos(t/2), s = sin(t/2); the adjoint uses -s.

template <int P>
__device__ __forceinline__ void rx_reg(St& a, float c, float s) {
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float xr = a.r[u], xi = a.i[u], yr = a.r[v], yi = a.i[v];
    // [c, -is; -is, c]
    a.r[u] = c * xr + s * yi;
    a.i[u] = c * xi - s * yr;
    a.r[v] = c * yr + s * xi;
    a.i[v] = c * yi - s * xr;
  }
}

template <int P>
__device__ __forceinline__ void ry_reg(St& a, float c, float s) {
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float xr = a.r[u], xi = a.i[u], yr = a.r[v], yi = a.i[v];
    // [c, -s; s, c]
    a.r[u] = c * xr - s * yr;
    a.i[u] = c * xi - s * yi;
    a.r[v] = s * xr + c * yr;
    a.i[v] = s * xi + c * yi;
  }
}

// diag(c - is, c + is) on register bit P
template <int P>
__device__ __forceinline__ void rz_reg(St& a, float c, float s) {
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const float ss = (u & (1 << P)) ? s : -s;
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = c * xr - ss * xi;
    a.i[u] = c * xi + ss * xr;
  }
}

// multiply every amplitude by (c + i ss)
__device__ __forceinline__ void phase_all(St& a, float c, float ss) {
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = c * xr - ss * xi;
    a.i[u] = c * xi + ss * xr;
  }
}

// CNOT with control and target on register bits: a register permutation
template <int C, int T>
__device__ __forceinline__ void cnot_rr(St& a) {
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (!(u & (1 << C)) || (u & (1 << T))) continue;
    const int v = u | (1 << T);
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = a.r[v];
    a.i[u] = a.i[v];
    a.r[v] = xr;
    a.i[v] = xi;
  }
}

// CNOT with the control on a thread bit (flag) and the target on register bit T
template <int T>
__device__ __forceinline__ void cnot_tr(St& a, bool flag) {
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (u & (1 << T)) continue;
    const int v = u | (1 << T);
    const float xr = a.r[u], xi = a.i[u], yr = a.r[v], yi = a.i[v];
    a.r[u] = flag ? yr : xr;
    a.i[u] = flag ? yi : xi;
    a.r[v] = flag ? xr : yr;
    a.i[v] = flag ? xi : yi;
  }
}

__device__ __forceinline__ uint32_t reg_pattern(int p) {
  return p == 0 ? 0xAAAAu : p == 1 ? 0xCCCCu : p == 2 ? 0xF0F0u : 0xFF00u;
}

// amplitudes whose register index u has bit u of `m` set are negated
__device__ __forceinline__ void negate_mask(St& a, uint32_t m) {
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const float sg = ((m >> u) & 1u) ? -1.f : 1.f;
    a.r[u] *= sg;
    a.i[u] *= sg;
  }
}

__device__ __forceinline__ void apply_rx(St& a, int p, float c, float s) {
  switch (p) {
    case 0: rx_reg<0>(a, c, s); break;
    case 1: rx_reg<1>(a, c, s); break;
    case 2: rx_reg<2>(a, c, s); break;
    default: rx_reg<3>(a, c, s); break;
  }
}

__device__ __forceinline__ void apply_ry(St& a, int p, float c, float s) {
  switch (p) {
    case 0: ry_reg<0>(a, c, s); break;
    case 1: ry_reg<1>(a, c, s); break;
    case 2: ry_reg<2>(a, c, s); break;
    default: ry_reg<3>(a, c, s); break;
  }
}

// RZ on physical bit p: register bit, or a thread bit (uniform phase per thread)
__device__ __forceinline__ void apply_rz(St& a, int p, float c, float s, int stid) {
  switch (p) {
    case 0: rz_reg<0>(a, c, s); break;
    case 1: rz_reg<1>(a, c, s); break;
    case 2: rz_reg<2>(a, c, s); break;
    case 3: rz_reg<3>(a, c, s); break;
    default: phase_all(a, c, ((stid >> (p - kRegBits)) & 1) ? s : -s); break;
  }
}

__device__ __forceinline__ void apply_cnot(St& a, int pc, int pt, int stid) {
  if (pc >= kRegBits) {
    const bool f = (stid >> (pc - kRegBits)) & 1;
    switch (pt) {
      case 0: cnot_tr<0>(a, f); break;
      case 1: cnot_tr<1>(a, f); break;
      case 2: cnot_tr<2>(a, f); break;
      default: cnot_tr<3>(a, f); break;
    }
    return;
  }
  switch (pc * 4 + pt) {
    case 1: cnot_rr<0, 1>(a); break;
    case 2: cnot_rr<0, 2>(a); break;
    case 3: cnot_rr<0, 3>(a); break;
    case 4: cnot_rr<1, 0>(a); break;
    case 6: cnot_rr<1, 2>(a); break;
    case 7: cnot_rr<1, 3>(a); break;
    case 8: cnot_rr<2, 0>(a); break;
    case 9: cnot_rr<2, 1>(a); break;
    case 11: cnot_rr<2, 3>(a); break;
    case 12: cnot_rr<3, 0>(a); break;
    case 13: cnot_rr<3, 1>(a); break;
    case 14: cnot_rr<3, 2>(a); break;
    default: break;
  }
}

__device__ __forceinline__ uint32_t bit_mask(int p, int stid) {
  if (p < kRegBits) return reg_pattern(p);
  return ((stid >> (p - kRegBits)) & 1) ? 0xFFFFu : 0u;
}

// ------------------------------------------------------- gradient partials
// Im(conj(l) p) = l.r p.i - l.i p.r ; Re(conj(l) p) = l.r p.r + l.i p.i

template <int P>
__device__ __forceinline__ float gx_reg(const St& l, const St& p) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    // X: <l|X|p> = conj(l0) p1 + conj(l1) p0
    acc += l.r[u] * p.i[v] - l.i[u] * p.r[v];
    acc += l.r[v] * p.i[u] - l.i[v] * p.r[u];
  }
  return acc;
}

template <int P>
__device__ __forceinline__ float gy_reg(const St& l, const St& p) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    // Y p = (-i p1, i p0): Im<l|Y|p> = -Re(conj(l0) p1) + Re(conj(l1) p0)
    acc -= l.r[u] * p.r[v] + l.i[u] * p.i[v];
    acc += l.r[v] * p.r[u] + l.i[v] * p.i[u];
  }
  return acc;
}

// Z on register bit P: sum over amplitudes of sign * Im(conj(l) p)
template <int P>
__device__ __forceinline__ float gz_reg(const St& l, const St& p) {
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const float v = l.r[u] * p.i[u] - l.i[u] * p.r[u];
    if (u & (1 << P)) a1 += v; else a0 += v;
  }
  return a0 - a1;
}

__device__ __forceinline__ float gz_all(const St& l, const St& p) {
  float a = 0.f;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) a += l.r[u] * p.i[u] - l.i[u] * p.r[u];
  return a;
}

__device__ __forceinline__ float grad_x(const St& l, const St& p, int r) {
  switch (r) {
    case 0: return gx_reg<0>(l, p);
    case 1: return gx_reg<1>(l, p);
    case 2: return gx_reg<2>(l, p);
    default: return gx_reg<3>(l, p);
  }
}

__device__ __forceinline__ float grad_y(const St& l, const St& p, int r) {
  switch (r) {
    case 0: return gy_reg<0>(l, p);
    case 1: return gy_reg<1>(l, p);
    case 2: return gy_reg<2>(l, p);
    default: return gy_reg<3>(l, p);
  }
}

__device__ __forceinline__ float grad_z(const St& l, const St& p, int ph, int stid) {
  switch (ph) {
    case 0: return gz_reg<0>(l, p);
    case 1: return gz_reg<1>(l, p);
    case 2: return gz_reg<2>(l, p);
    case 3: return gz_reg<3>(l, p);
    default: {
      const float v = gz_all(l, p);
      return ((stid >> (ph - kRegBits)) & 1) ? -v : v;
    }
  }
}

// --------------------------------------------------------------- helpers

// butterfly sum over `width` consecutive lanes (power of two <= 64); every lane
// of the segment ends with the same, order-fixed value
__device__ __forceinline__ float seg_sum(float v, int width) {
  for (int m = 1; m < width; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// LDS exchange: write the 16 amplitudes at lam(old index), read lam(new index).
// col[0..k) are the write-side columns, col[k..2k) the read-side columns.
__device__ __forceinline__ void exchange(St& a, float2* xbuf, const uint32_t* col, int k, int t,
                                         int stid, int sl) {
  uint32_t bw = 0, br = 0;
  for (int i = 0; i < t; ++i) {
    if ((stid >> i) & 1) {
      bw ^= col[kRegBits + i];
      br ^= col[k + kRegBits + i];
    }
  }
  // samples sharing a 32-lane group are spread over different banks
  const uint32_t lowmask = (1u << (k < kBankBits ? k : kBankBits)) - 1u;
  const uint32_t xs = ((uint32_t)sl << t) & lowmask;
  const uint32_t base = (uint32_t)sl << k;
  bw = base | (bw ^ xs);
  br = base | (br ^ xs);
  const uint32_t w0 = col[0], w1 = col[1], w2 = col[2], w3 = col[3];
  const uint32_t r0 = col[k], r1 = col[k + 1], r2 = col[k + 2], r3 = col[k + 3];
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const uint32_t o = ((u & 1) ? w0 : 0u) ^ ((u & 2) ? w1 : 0u) ^ ((u & 4) ? w2 : 0u) ^
                       ((u & 8) ? w3 : 0u);
    xbuf[bw ^ o] = make_float2(a.r[u], a.i[u]);
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const uint32_t o = ((u & 1) ? r0 : 0u) ^ ((u & 2) ? r1 : 0u) ^ ((u & 4) ? r2 : 0u) ^
                       ((u & 8) ? r3 : 0u);
    const float2 v = xbuf[br ^ o];
    a.r[u] = v.x;
    a.i[u] = v.y;
  }
  __syncthreads();
}

// ------------------------------------------------------------------ kernel

template <int WG, bool BWD>
__global__ void __launch_bounds__(WG) resident_kernel(const TileArgs A) {
  extern __shared__ __align__(16) unsigned char smem[];
  float2* xbuf = reinterpret_cast<float2*>(smem);
  float2* tab = reinterpret_cast<float2*>(smem + A.lds_tab);
  float* acc = reinterpret_cast<float*>(smem + A.lds_acc);

  const int tid = threadIdx.x;
  const int T = 1 << A.t;
  const int stid = tid & (T - 1);
  const int sl = tid >> A.t;
  const int S = A.S;
  const int64_t b0 = (int64_t)blockIdx.x * S;
  const int64_t b = b0 + sl;
  const bool valid = b < A.B;
  const int width = T < 64 ? T : 64;
  const int grp = T < 64 ? sl : (tid >> 6);
  const bool leader = (tid & (width - 1)) == 0;

  // 1. parameter resolution: (cos, sin)(theta / 2) per occurrence and sample
  for (int i = tid; i < A.n_occ * S; i += WG) {
    const int o = i / S;
    const int s = i - o * S;
    const int64_t bb = b0 + s;
    const int src = A.occ_src[o];
    float c, sn;
    if (src == VQC_SRC_CONST) {
      c = A.occ_cs[2 * o];
      sn = A.occ_cs[2 * o + 1];
    } else {
      float th = 0.f;
      if (bb < A.B)
        th = src == VQC_SRC_PARAM ? A.params[bb * A.P + A.occ_idx[o]]
                                  : A.inputs[bb * A.F + A.occ_idx[o]];
      sincosf(0.5f * th, &sn, &c);
    }
    tab[i] = make_float2(c, sn);
  }
  if (BWD)
    for (int i = tid; i < A.n_slots * A.G; i += WG) acc[i] = 0.f;
  __syncthreads();

  // 2. state
  St a, l;
  if (!BWD) {
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) {
      a.r[j] = 0.f;
      a.i[j] = 0.f;
    }
    if (stid == 0) a.r[0] = 1.f;
  } else {
    const float2* ws = reinterpret_cast<const float2*>(A.ws);
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) {
      const float2 v = ws[((size_t)blockIdx.x * kRegAmps + j) * WG + tid];
      a.r[j] = v.x;
      a.i[j] = v.y;
    }
    // lambda = H psi_G, H = sum_q g_q Z_q
    float gt = 0.f, g0 = 0.f, g1 = 0.f, g2 = 0.f, g3 = 0.f;
    if (valid) {
      for (int q = 0; q < A.n; ++q) {
        const float gq = A.grad_out[b * A.n + q];
        const int p = A.end_phys[q];
        if (p == 0) g0 += gq;
        else if (p == 1) g1 += gq;
        else if (p == 2) g2 += gq;
        else if (p == 3) g3 += gq;
        else gt += ((stid >> (p - kRegBits)) & 1) ? -gq : gq;
      }
    }
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) {
      const float h = gt + ((j & 1) ? -g0 : g0) + ((j & 2) ? -g1 : g1) + ((j & 4) ? -g2 : g2) +
                      ((j & 8) ? -g3 : g3);
      l.r[j] = h * a.r[j];
      l.i[j] = h * a.i[j];
    }
  }

  // 3. the schedule
  for (int pc = 0; pc < A.n_ins; ++pc) {
    const uint32_t w0 = A.ins[2 * pc];
    const uint32_t arg = A.ins[2 * pc + 1];
    const int op = w0 & 255;
    const int pa = (w0 >> 8) & 255;
    const int pb = (w0 >> 16) & 255;
    if (op == OP_EXCHANGE) {
      exchange(a, xbuf, A.cols + arg, A.k, A.t, stid, sl);
      if (BWD) exchange(l, xbuf, A.cols + arg, A.k, A.t, stid, sl);
      continue;
    }
    if (op == OP_CNOT) {
      apply_cnot(a, pa, pb, stid);
      if (BWD) apply_cnot(l, pa, pb, stid);
      continue;
    }
    if (op == OP_CZ) {
      const uint32_t m = bit_mask(pa, stid) & bit_mask(pb, stid);
      negate_mask(a, m);
      if (BWD) negate_mask(l, m);
      continue;
    }
    const float2 cs = tab[arg * S + sl];
    if (!BWD) {
      if (op == OP_RX) apply_rx(a, pa, cs.x, cs.y);
      else if (op == OP_RY) apply_ry(a, pa, cs.x, cs.y);
      else apply_rz(a, pa, cs.x, cs.y, stid);
    } else {
      float g;
      if (op == OP_RX) {
        g = grad_x(l, a, pa);
        apply_rx(a, pa, cs.x, -cs.y);
        apply_rx(l, pa, cs.x, -cs.y);
      } else if (op == OP_RY) {
        g = grad_y(l, a, pa);
        apply_ry(a, pa, cs.x, -cs.y);
        apply_ry(l, pa, cs.x, -cs.y);
      } else {
        g = grad_z(l, a, pa, stid);
        apply_rz(a, pa, cs.x, -cs.y, stid);
        apply_rz(l, pa, cs.x, -cs.y, stid);
      }
      g = seg_sum(g, width);
      const int slot = A.occ_slot[arg];
      if (slot >= 0 && leader) atomicAdd(&acc[slot * A.G + grp], g);
    }
  }

  // 4. epilogue
  if (!BWD) {
    if (A.ws) {
      float2* ws = reinterpret_cast<float2*>(A.ws);
#pragma unroll
      for (int j = 0; j < kRegAmps; ++j)
        ws[((size_t)blockIdx.x * kRegAmps + j) * WG + tid] = make_float2(a.r[j], a.i[j]);
    }
    float tot = 0.f, s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) {
      const float pj = a.r[j] * a.r[j] + a.i[j] * a.i[j];
      tot += pj;
      s0 += (j & 1) ? -pj : pj;
      s1 += (j & 2) ? -pj : pj;
      s2 += (j & 4) ? -pj : pj;
      s3 += (j & 8) ? -pj : pj;
    }
    float* ez = reinterpret_cast<float*>(xbuf);  // the exchange buffer is idle now
    __syncthreads();
    for (int q = 0; q < A.n; ++q) {
      const int p = A.end_phys[q];
      float v;
      if (p == 0) v = s0;
      else if (p == 1) v = s1;
      else if (p == 2) v = s2;
      else if (p == 3) v = s3;
      else v = ((stid >> (p - kRegBits)) & 1) ? -tot : tot;
      v = seg_sum(v, width);
      if (leader) ez[q * A.G + grp] = v;
    }
    __syncthreads();
    for (int i = tid; i < A.n * S; i += WG) {
      const int q = i / S;
      const int s = i - q * S;
      const int64_t bb = b0 + s;
      if (bb >= A.B) continue;
      float e;
      if (T >= 64) {
        e = 0.f;
        for (int g = 0; g < A.G; ++g) e += ez[q * A.G + g];
      } else {
        e = ez[q * A.G + s];
      }
      A.expvals[bb * A.n + q] = e;
    }
  } else {
    __syncthreads();
    for (int i = tid; i < A.n_slots * S; i += WG) {
      const int slot = i / S;
      const int s = i - slot * S;
      const int64_t bb = b0 + s;
      if (bb >= A.B) continue;
      float v;
      if (T >= 64) {
        v = 0.f;
        for (int g = 0; g < A.G; ++g) v += acc[slot * A.G + g];
      } else {
        v = acc[slot * A.G + s];
      }
      if (slot < A.P) {
        if (A.dparams) A.dparams[bb * A.P + slot] = v;
      } else if (A.dinputs) {
        A.dinputs[bb * A.F + (slot - A.P)] = v;
      }
    }
  }
}

__global__ void loss_grad_kernel(int kind, int64_t B, int n, const float* __restrict__ e,
                                 const float* __restrict__ y, float* __restrict__ g) {
  const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const float* eb = e + b * n;
  float* gb = g + b * n;
  switch (kind) {
    case VQC_LOSS_SUM:
      for (int j = 0; j < n; ++j) gb[j] = 1.f;
      break;
    case VQC_LOSS_MEAN:
      for (int j = 0; j < n; ++j) gb[j] = 1.f / (float)n;
      break;
    case VQC_LOSS_MSE_Z0:
      gb[0] = 2.f * (eb[0] - y[b]) / (float)B;
      for (int j = 1; j < n; ++j) gb[j] = 0.f;
      break;
    default: {
      float s = 0.f;
      for (int j = 0; j < n; ++j) s += eb[j];
      s /= (float)n;
      const float v = 2.f * (s - y[b]) / ((float)n * (float)B);
      for (int j = 0; j < n; ++j) gb[j] = v;
    }
  }
}

template <int WG, bool BWD>
int launch_wg(const TileArgs& a, int64_t blocks, size_t lds, void* stream) {
  hipLaunchKernelGGL((resident_kernel<WG, BWD>), dim3((unsigned)blocks), dim3(WG), lds,
                     (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

template <bool BWD>
int launch_any(int wg, const TileArgs& a, int64_t blocks, size_t lds, void* stream) {
  switch (wg) {
    case 64: return launch_wg<64, BWD>(a, blocks, lds, stream);
    case 128: return launch_wg<128, BWD>(a, blocks, lds, stream);
    case 256: return launch_wg<256, BWD>(a, blocks, lds, stream);
    case 512: return launch_wg<512, BWD>(a, blocks, lds, stream);
    case 1024: return launch_wg<1024, BWD>(a, blocks, lds, stream);
    default: return (int)hipErrorInvalidValue;
  }
}

template <int WG>
int set_lds(size_t f, size_t b) {
  hipError_t e1 = hipFuncSetAttribute((const void*)resident_kernel<WG, false>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)f);
  hipError_t e2 = hipFuncSetAttribute((const void*)resident_kernel<WG, true>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)b);
  return (int)(e1 != hipSuccess ? e1 : e2);
}

}  // namespace

int prepare_kernels(int wg, size_t lds_fwd, size_t lds_bwd) {
  switch (wg) {
    case 64: return set_lds<64>(lds_fwd, lds_bwd);
    case 128: return set_lds<128>(lds_fwd, lds_bwd);
    case 256: return set_lds<256>(lds_fwd, lds_bwd);
    case 512: return set_lds<512>(lds_fwd, lds_bwd);
    case 1024: return set_lds<1024>(lds_fwd, lds_bwd);
    default: return (int)hipErrorInvalidValue;
  }
}

int launch_resident_forward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream) {
  return launch_any<false>(plan.WG, a, blocks, plan.lds_fwd, stream);
}

int launch_resident_backward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream) {
  return launch_any<true>(plan.WG, a, blocks, plan.lds_bwd, stream);
}

int launch_loss_grad(int kind, int64_t batch, int n, const float* e, const float* y, float* g,
                     void* stream) {
  const int threads = 256;
  const int64_t blocks = (batch + threads - 1) / threads;
  hipLaunchKernelGGL(loss_grad_kernel, dim3((unsigned)blocks), dim3(threads), 0,
                     (hipStream_t)stream, kind, batch, n, e, y, g);
  return (int)hipGetLastError();
}

}  // namespace vqc
