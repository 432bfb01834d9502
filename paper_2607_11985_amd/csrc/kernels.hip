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
__device__ __forceinline__ void apply_rz(St& a, int p, float c, float s, uint32_t tb) {
  switch (p) {
    case 0: rz_reg<0>(a, c, s); break;
    case 1: rz_reg<1>(a, c, s); break;
    case 2: rz_reg<2>(a, c, s); break;
    case 3: rz_reg<3>(a, c, s); break;
    default: phase_all(a, c, ((tb >> (p - kRegBits)) & 1u) ? s : -s); break;
  }
}

__device__ __forceinline__ void apply_cnot(St& a, int pc, int pt, uint32_t tb) {
  if (pc >= kRegBits) {
    const bool f = (tb >> (pc - kRegBits)) & 1u;
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

// tb: the bits of the amplitude position above the register bits (thread index
// within the tile, then the tile index of a streamed sample)
__device__ __forceinline__ uint32_t bit_mask(int p, uint32_t tb) {
  if (p < kRegBits) return reg_pattern(p);
  return ((tb >> (p - kRegBits)) & 1u) ? 0xFFFFu : 0u;
}

// ------------------------------------------- fused adjoint rotation steps
// One pass over the amplitude pairs: accumulate dL/dtheta = Im <l| P |a> and
// un-apply R_P(theta) (i.e. apply R_P(-theta)) to both a and l.  Working pair by
// pair keeps only the pair's old values alive.

template <int P>
__device__ __forceinline__ float adj_rx(St& a, St& l, float c, float s) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float ar = a.r[u], ai = a.i[u], br = a.r[v], bi = a.i[v];
    const float lr = l.r[u], li = l.i[u], mr = l.r[v], mi = l.i[v];
    // X: <l|X|a> = conj(l0) a1 + conj(l1) a0
    acc += lr * bi - li * br;
    acc += mr * ai - mi * ar;
    // RX(-theta) = [c, is; is, c]
    a.r[u] = c * ar - s * bi;
    a.i[u] = c * ai + s * br;
    a.r[v] = c * br - s * ai;
    a.i[v] = c * bi + s * ar;
    l.r[u] = c * lr - s * mi;
    l.i[u] = c * li + s * mr;
    l.r[v] = c * mr - s * li;
    l.i[v] = c * mi + s * lr;
  }
  return acc;
}

template <int P>
__device__ __forceinline__ float adj_ry(St& a, St& l, float c, float s) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float ar = a.r[u], ai = a.i[u], br = a.r[v], bi = a.i[v];
    const float lr = l.r[u], li = l.i[u], mr = l.r[v], mi = l.i[v];
    // Y a = (-i a1, i a0): Im<l|Y|a> = -Re(conj(l0) a1) + Re(conj(l1) a0)
    acc -= lr * br + li * bi;
    acc += mr * ar + mi * ai;
    // RY(-theta) = [c, s; -s, c]
    a.r[u] = c * ar + s * br;
    a.i[u] = c * ai + s * bi;
    a.r[v] = c * br - s * ar;
    a.i[v] = c * bi - s * ai;
    l.r[u] = c * lr + s * mr;
    l.i[u] = c * li + s * mi;
    l.r[v] = c * mr - s * lr;
    l.i[v] = c * mi - s * li;
  }
  return acc;
}

// RZ on register bit P: Im<l|Z|a> and diag(c + is, c - is) on both states
template <int P>
__device__ __forceinline__ float adj_rz(St& a, St& l, float c, float s) {
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const float ar = a.r[u], ai = a.i[u], lr = l.r[u], li = l.i[u];
    const float v = lr * ai - li * ar;
    if (u & (1 << P)) a1 += v; else a0 += v;
    const float ss = (u & (1 << P)) ? -s : s;  // the inverse phase
    a.r[u] = c * ar - ss * ai;
    a.i[u] = c * ai + ss * ar;
    l.r[u] = c * lr - ss * li;
    l.i[u] = c * li + ss * lr;
  }
  return a0 - a1;
}

// RZ on a thread / global bit: the Z sign and the inverse phase are uniform
__device__ __forceinline__ float adj_rz_uniform(St& a, St& l, float c, float s, bool one) {
  float acc = 0.f;
  const float ss = one ? -s : s;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const float ar = a.r[u], ai = a.i[u], lr = l.r[u], li = l.i[u];
    acc += lr * ai - li * ar;
    a.r[u] = c * ar - ss * ai;
    a.i[u] = c * ai + ss * ar;
    l.r[u] = c * lr - ss * li;
    l.i[u] = c * li + ss * lr;
  }
  return one ? -acc : acc;
}

__device__ __forceinline__ float adjoint_rotation(int op, St& a, St& l, int p, float c, float s,
                                                  uint32_t tb) {
  if (op == OP_RX) {
    switch (p) {
      case 0: return adj_rx<0>(a, l, c, s);
      case 1: return adj_rx<1>(a, l, c, s);
      case 2: return adj_rx<2>(a, l, c, s);
      default: return adj_rx<3>(a, l, c, s);
    }
  }
  if (op == OP_RY) {
    switch (p) {
      case 0: return adj_ry<0>(a, l, c, s);
      case 1: return adj_ry<1>(a, l, c, s);
      case 2: return adj_ry<2>(a, l, c, s);
      default: return adj_ry<3>(a, l, c, s);
    }
  }
  switch (p) {
    case 0: return adj_rz<0>(a, l, c, s);
    case 1: return adj_rz<1>(a, l, c, s);
    case 2: return adj_rz<2>(a, l, c, s);
    case 3: return adj_rz<3>(a, l, c, s);
    default: return adj_rz_uniform(a, l, c, s, (tb >> (p - kRegBits)) & 1u);
  }
}

// --------------------------------------------------------------- helpers

// Stores a loaded (re, im) pair into two independent 32-bit values.  Without
// the empty asm the pair stays one 64-bit register tuple whose halves are later
// rewritten separately, and the allocator then keeps (and spills) dead halves.
__device__ __forceinline__ void split(const float2 v, float& r, float& i) {
  float x = v.x, y = v.y;
  asm volatile("" : "+v"(x), "+v"(y));
  r = x;
  i = y;
}


// butterfly sum over `width` consecutive lanes (power of two <= 64); every lane
// of the segment ends with the same, order-fixed value
__device__ __forceinline__ float seg_sum(float v, int width) {
  for (int m = 1; m < width; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// the same over the whole wave, fully unrolled
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// LDS exchange: write the 16 amplitudes at lam(old index), read lam(new index).
// col[0..k) are the write-side columns, col[k..2k) the read-side columns.  The
// buffer is planar (real parts, then imaginary parts, `plane` floats apart) so
// every access is a 32-bit one: no 64-bit register tuples enter the schedule
// loop, and 32 lanes hit 32 banks.
__device__ __forceinline__ void exchange(St& a, float* xbuf, uint32_t plane, const uint32_t* col,
                                         int k, int t, int stid, int sl) {
  uint32_t bw = 0, br = 0;
#pragma unroll
  for (int i = 0; i < kMaxTileQubits - kRegBits; ++i) {
    if (i < t && ((stid >> i) & 1)) {
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
  float* xr = xbuf;
  float* xi = xbuf + plane;
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const uint32_t o = ((u & 1) ? w0 : 0u) ^ ((u & 2) ? w1 : 0u) ^ ((u & 4) ? w2 : 0u) ^
                       ((u & 8) ? w3 : 0u);
    xr[bw ^ o] = a.r[u];
    xi[bw ^ o] = a.i[u];
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kRegAmps; ++u) {
    const uint32_t o = ((u & 1) ? r0 : 0u) ^ ((u & 2) ? r1 : 0u) ^ ((u & 4) ? r2 : 0u) ^
                       ((u & 8) ? r3 : 0u);
    a.r[u] = xr[br ^ o];
    a.i[u] = xi[br ^ o];
  }
  __syncthreads();
}

// ------------------------------------------------------- schedule runner

// Context of one workgroup's walk through an instruction stream.
struct Walk {
  const uint32_t* cols;
  float* xbuf;        // planar exchange buffer: plane floats of real parts, then imaginary
  uint32_t plane;
  const float2* tab;  // (cos, sin)(theta/2), [occurrence][S]
  float* acc;         // gradient accumulators [slot][G]
  int k, t, S, G;
  int stid, sl, grp, width;
  uint32_t tb;        // tile bits above the register bits
  bool leader;
};

// Runs `n_ins` instructions on psi (a) and, for the adjoint, lambda (l).
// WIDE: every sample spans whole waves (the reduction width is 64).
template <bool BWD, bool WIDE>
__device__ __forceinline__ void run_schedule(St& a, St& l, const uint32_t* ins, int n_ins,
                                             const Walk& w) {
  for (int pc = 0; pc < n_ins; ++pc) {
    const uint32_t w0 = ins[2 * pc];
    const uint32_t arg = ins[2 * pc + 1];
    const int op = w0 & 31;
    const int pa = (w0 >> 5) & 31;
    const int pb = (w0 >> 10) & 31;
    if (op == OP_EXCHANGE) {
      exchange(a, w.xbuf, w.plane, w.cols + arg, w.k, w.t, w.stid, w.sl);
      if (BWD) exchange(l, w.xbuf, w.plane, w.cols + arg, w.k, w.t, w.stid, w.sl);
      continue;
    }
    if (op == OP_CNOT) {
      apply_cnot(a, pa, pb, w.tb);
      if (BWD) apply_cnot(l, pa, pb, w.tb);
      continue;
    }
    if (op == OP_CZ) {
      const uint32_t m = bit_mask(pa, w.tb) & bit_mask(pb, w.tb);
      negate_mask(a, m);
      if (BWD) negate_mask(l, m);
      continue;
    }
    const float2 cs = w.tab[arg * w.S + w.sl];
    if (!BWD) {
      if (op == OP_RX) apply_rx(a, pa, cs.x, cs.y);
      else if (op == OP_RY) apply_ry(a, pa, cs.x, cs.y);
      else apply_rz(a, pa, cs.x, cs.y, w.tb);
    } else {
      // dL/dtheta = Im <lambda| P |psi>, then psi, lambda <- R(-theta) psi, lambda
      float g = adjoint_rotation(op, a, l, pa, cs.x, cs.y, w.tb);
      const int slot = (int)(w0 >> 16) - 1;
      g = WIDE ? wave_sum(g) : seg_sum(g, w.width);
      if (slot >= 0 && w.leader) atomicAdd(&w.acc[slot * w.G + w.grp], g);
    }
  }
}

// Parameter resolution: (cos, sin)(theta/2) for every occurrence and sample of
// the workgroup.  Constant angles come precomputed from the compile phase.
__device__ __forceinline__ void angle_table(float2* tab, int n_occ, int S, int64_t b0, int64_t B,
                                            const int32_t* occ_src, const int32_t* occ_idx,
                                            const float* occ_cs, const float* params, int P,
                                            const float* inputs, int F, int tid, int nthreads) {
  for (int i = tid; i < n_occ * S; i += nthreads) {
    const int o = i / S;
    const int s = i - o * S;
    const int64_t bb = b0 + s;
    const int src = occ_src[o];
    float c, sn;
    if (src == VQC_SRC_CONST) {
      c = occ_cs[2 * o];
      sn = occ_cs[2 * o + 1];
    } else {
      float th = 0.f;
      if (bb < B)
        th = src == VQC_SRC_PARAM ? params[bb * P + occ_idx[o]] : inputs[bb * F + occ_idx[o]];
      sincosf(0.5f * th, &sn, &c);
    }
    tab[i] = make_float2(c, sn);
  }
}

// lambda = H psi with H = sum_q g_q Z_q, the Z signs read from the mapping
__device__ __forceinline__ void make_lambda(St& l, const St& a, const float* g, int n,
                                            const uint8_t* phys, uint32_t tb, bool valid) {
  float gt = 0.f, g0 = 0.f, g1 = 0.f, g2 = 0.f, g3 = 0.f;
  if (valid) {
    for (int q = 0; q < n; ++q) {
      const float gq = g[q];
      const int p = phys[q];
      if (p == 0) g0 += gq;
      else if (p == 1) g1 += gq;
      else if (p == 2) g2 += gq;
      else if (p == 3) g3 += gq;
      else gt += ((tb >> (p - kRegBits)) & 1u) ? -gq : gq;
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

// Per-qubit signed probability sums of this workgroup's amplitudes:
// ez[q * G + grp] = sum over the group's amplitudes of (-1)^{x_q} |a|^2.
// Must be called by every thread; ez may alias the exchange buffer.
__device__ __forceinline__ void z_partials(const St& a, float* ez, int n, const uint8_t* phys,
                                           const Walk& w) {
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
  __syncthreads();  // the exchange buffer may still be read by other threads
  for (int q = 0; q < n; ++q) {
    const int p = phys[q];
    float v;
    if (p == 0) v = s0;
    else if (p == 1) v = s1;
    else if (p == 2) v = s2;
    else if (p == 3) v = s3;
    else v = ((w.tb >> (p - kRegBits)) & 1u) ? -tot : tot;
    v = seg_sum(v, w.width);
    if (w.leader) ez[q * w.G + w.grp] = v;
  }
  __syncthreads();
}

// ------------------------------------------------------ resident kernel

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
  Walk w;
  w.cols = A.cols;
  w.xbuf = reinterpret_cast<float*>(xbuf);
  w.plane = (uint32_t)WG * kRegAmps;
  w.tab = tab;
  w.acc = acc;
  w.k = A.k;
  w.t = A.t;
  w.S = S;
  w.G = A.G;
  w.stid = stid;
  w.sl = sl;
  w.width = T < 64 ? T : 64;
  w.grp = T < 64 ? sl : (tid >> 6);
  w.leader = (tid & (w.width - 1)) == 0;
  w.tb = (uint32_t)stid;

  angle_table(tab, A.n_occ, S, b0, A.B, A.occ_src, A.occ_idx, A.occ_cs, A.params, A.P, A.inputs,
              A.F, tid, WG);
  if (BWD)
    for (int i = tid; i < A.n_slots * A.G; i += WG) acc[i] = 0.f;
  __syncthreads();

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
      split(ws[((size_t)blockIdx.x * kRegAmps + j) * WG + tid], a.r[j], a.i[j]);
    }
    make_lambda(l, a, A.grad_out + (valid ? b : 0) * A.n, A.n, A.end_phys, w.tb, valid);
  }

  if (WG > 64) run_schedule<BWD, true>(a, l, A.ins, A.n_ins, w);
  else run_schedule<BWD, false>(a, l, A.ins, A.n_ins, w);

  if (!BWD) {
    if (A.ws) {
      float2* ws = reinterpret_cast<float2*>(A.ws);
#pragma unroll
      for (int j = 0; j < kRegAmps; ++j)
        ws[((size_t)blockIdx.x * kRegAmps + j) * WG + tid] = make_float2(a.r[j], a.i[j]);
    }
    float* ez = reinterpret_cast<float*>(xbuf);
    z_partials(a, ez, A.n, A.end_phys, w);
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

// ----------------------------------------------------- streaming kernel
// One pass over B * 2^ng tiles of 2^14 amplitudes (1024 threads x 16).  Tiles
// are read and written in the pass's I/O layout: tile rank r (the position of
// an amplitude among the 14 local qubits in ascending order) has r = stid +
// 1024 j, so consecutive lanes touch consecutive low-qubit addresses.

constexpr int kStreamWG = 1 << (kMaxTileQubits - kRegBits);

__device__ __forceinline__ void io_offsets(const uint32_t* io, int k, int ng, int stid, int g,
                                           uint32_t& base, uint32_t (&off)[kRegAmps]) {
  const int nt = k - kRegBits;
  base = 0;
  for (int i = 0; i < nt; ++i)
    if ((stid >> i) & 1) base |= io[i];
  for (int i = 0; i < ng; ++i)
    if ((g >> i) & 1) base |= io[k + i];
  const uint32_t c0 = io[nt], c1 = io[nt + 1], c2 = io[nt + 2], c3 = io[nt + 3];
#pragma unroll
  for (int j = 0; j < kRegAmps; ++j)
    off[j] = ((j & 1) ? c0 : 0u) | ((j & 2) ? c1 : 0u) | ((j & 4) ? c2 : 0u) | ((j & 8) ? c3 : 0u);
}

template <bool BWD>
__global__ void __launch_bounds__(kStreamWG) stream_kernel(const PassArgs A) {
  extern __shared__ __align__(16) unsigned char smem[];
  float2* xbuf = reinterpret_cast<float2*>(smem);
  float2* tab = reinterpret_cast<float2*>(smem + A.lds_tab);
  float* acc = reinterpret_cast<float*>(smem + A.lds_acc);
  const int tid = threadIdx.x;
  const int64_t blk = blockIdx.x;
  const int64_t b = blk >> A.ng;
  const int g = (int)(blk & ((1 << A.ng) - 1));
  constexpr int G = kStreamWG / 64;
  Walk w;
  w.cols = A.cols;
  w.xbuf = reinterpret_cast<float*>(xbuf);
  w.plane = (uint32_t)kStreamWG * kRegAmps;
  w.tab = tab;
  w.acc = acc;
  w.k = A.k;
  w.t = A.k - kRegBits;
  w.S = 1;
  w.G = G;
  w.stid = tid;
  w.sl = 0;
  w.width = 64;
  w.grp = tid >> 6;
  w.leader = (tid & 63) == 0;
  w.tb = (uint32_t)tid | ((uint32_t)g << w.t);

  angle_table(tab, A.n_occ, 1, b, A.B, A.occ_src, A.occ_idx, A.occ_cs, A.params, A.P, A.inputs,
              A.F, tid, kStreamWG);
  if (BWD)
    for (int i = tid; i < A.n_pslots * G; i += kStreamWG) acc[i] = 0.f;
  __syncthreads();

  uint32_t base, off[kRegAmps];
  io_offsets(A.io, A.k, A.ng, tid, g, base, off);
  const size_t sbase = (size_t)b << (A.k + A.ng);
  St a, l;
  if (!BWD && (A.flags & PF_INIT)) {
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) {
      a.r[j] = 0.f;
      a.i[j] = 0.f;
    }
    if (tid == 0 && g == 0) a.r[0] = 1.f;
  } else {
    const float2* src = reinterpret_cast<const float2*>(A.psi_src) + sbase;
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) split(src[base | off[j]], a.r[j], a.i[j]);
  }
  if (BWD) {
    if (A.flags & PF_MAKE_LAMBDA) {
      make_lambda(l, a, A.grad_out + b * A.n, A.n, A.start_phys, w.tb, true);
    } else {
      const float2* src = reinterpret_cast<const float2*>(A.lam_src) + sbase;
#pragma unroll
      for (int j = 0; j < kRegAmps; ++j) split(src[base | off[j]], l.r[j], l.i[j]);
    }
  }

  run_schedule<BWD, true>(a, l, A.ins, A.n_ins, w);

  // recompute the I/O offsets instead of keeping them alive through the schedule
  int tid2 = tid;
  asm volatile("" : "+v"(tid2));
  io_offsets(A.io, A.k, A.ng, tid2, g, base, off);
  {
    float2* dst = reinterpret_cast<float2*>(A.psi_dst) + sbase;
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) dst[base | off[j]] = make_float2(a.r[j], a.i[j]);
  }
  if (BWD) {
    float2* dst = reinterpret_cast<float2*>(A.lam_dst) + sbase;
#pragma unroll
    for (int j = 0; j < kRegAmps; ++j) dst[base | off[j]] = make_float2(l.r[j], l.i[j]);
    __syncthreads();
    float* gp = A.gpart + blk * A.n_slots;
    for (int i = tid; i < A.n_pslots; i += kStreamWG) {
      float v = 0.f;
      for (int r = 0; r < G; ++r) v += acc[i * G + r];
      gp[A.pslots[i]] += v;
    }
  } else if (A.flags & PF_ZPART) {
    float* ez = reinterpret_cast<float*>(xbuf);
    z_partials(a, ez, A.n, A.end_phys, w);
    for (int q = tid; q < A.n; q += kStreamWG) {
      float e = 0.f;
      for (int r = 0; r < G; ++r) e += ez[q * G + r];
      A.epart[blk * A.n + q] = e;
    }
  }
}

__global__ void reduce_e_kernel(int64_t B, int ng, int n, const float* __restrict__ epart,
                                float* __restrict__ e) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * n) return;
  const int64_t b = i / n;
  const int q = (int)(i - b * n);
  float v = 0.f;
  for (int g = 0; g < (1 << ng); ++g) v += epart[((b << ng) + g) * n + q];
  e[i] = v;
}

__global__ void reduce_grad_kernel(int64_t B, int ng, int n_slots, int P, int F,
                                   const float* __restrict__ gpart, float* __restrict__ dparams,
                                   float* __restrict__ dinputs) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * n_slots) return;
  const int64_t b = i / n_slots;
  const int s = (int)(i - b * n_slots);
  float v = 0.f;
  for (int g = 0; g < (1 << ng); ++g) v += gpart[((b << ng) + g) * n_slots + s];
  if (s < P) {
    if (dparams) dparams[b * P + s] = v;
  } else if (dinputs) {
    dinputs[b * F + (s - P)] = v;
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0.f;
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

unsigned grid_1d(int64_t count, int threads) { return (unsigned)((count + threads - 1) / threads); }

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

int prepare_stream_kernels(size_t lds_fwd, size_t lds_bwd) {
  hipError_t e1 = hipFuncSetAttribute((const void*)stream_kernel<false>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_fwd);
  hipError_t e2 = hipFuncSetAttribute((const void*)stream_kernel<true>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bwd);
  return (int)(e1 != hipSuccess ? e1 : e2);
}

int launch_resident_forward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream) {
  return launch_any<false>(plan.WG, a, blocks, plan.lds_fwd, stream);
}

int launch_resident_backward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream) {
  return launch_any<true>(plan.WG, a, blocks, plan.lds_bwd, stream);
}

int launch_stream_pass(bool bwd, const PassArgs& a, int64_t blocks, size_t lds, void* stream) {
  if (bwd)
    hipLaunchKernelGGL(stream_kernel<true>, dim3((unsigned)blocks), dim3(kStreamWG), lds,
                       (hipStream_t)stream, a);
  else
    hipLaunchKernelGGL(stream_kernel<false>, dim3((unsigned)blocks), dim3(kStreamWG), lds,
                       (hipStream_t)stream, a);
  return (int)hipGetLastError();
}

int launch_reduce_e(int64_t batch, int ng, int n, const float* epart, float* e, void* stream) {
  hipLaunchKernelGGL(reduce_e_kernel, dim3(grid_1d(batch * n, 256)), dim3(256), 0,
                     (hipStream_t)stream, batch, ng, n, epart, e);
  return (int)hipGetLastError();
}

int launch_reduce_grad(int64_t batch, int ng, int n_slots, int P, int F, const float* gpart,
                       float* dparams, float* dinputs, void* stream) {
  if (batch * n_slots == 0) return 0;
  hipLaunchKernelGGL(reduce_grad_kernel, dim3(grid_1d(batch * n_slots, 256)), dim3(256), 0,
                     (hipStream_t)stream, batch, ng, n_slots, P, F, gpart, dparams, dinputs);
  return (int)hipGetLastError();
}

int launch_fill_zero(float* p, int64_t count, void* stream) {
  if (count == 0) return 0;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_1d(count, 256)), dim3(256), 0,
                     (hipStream_t)stream, p, count);
  return (int)hipGetLastError();
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
