// vqc_device.h -- device code of the batched VQC engine for gfx950, shared by
// the precompiled kernels (kernels.hip) and by the kernels generated and
// compiled at run time for one specific circuit.
//
// Register tile: a workgroup keeps a tile of 2^k amplitudes on chip, 2^R per
// thread (R register bits), for the whole circuit (Algorithm 1, execute phase):
//   1. per-sample angle table: (cos, sin)(theta/2) for every rotation
//      occurrence, theta read from params / inputs, constants from the
//      compiled schedule (parameter resolution);
//   2. state init |0...0> in registers, or a tile loaded from HBM;
//   3. the schedule: register-bit rotations and CNOTs (VALU only), diagonal RZ
//      / CZ on any bit, LDS exchanges that move other qubits onto the register
//      bits;
//   4. epilogue: <Z_j> partial sums (Algorithm 1, return statement), tile
//      store, gradient sums.
// The adjoint kernels start from psi_G, form lambda = (sum_j g_j Z_j) psi_G
// and walk the schedule backwards: for every rotation R_P(t) they accumulate
// dL/dt = Im <lambda| P |psi> and un-apply the gate on both states
// (psi <- U^dagger psi, lambda <- U^dagger lambda): the exact gradient of
// Sec. 3 "Gate Application and Differentiation" with O(state) memory.
#pragma once
#include "vqc_structs.h"

namespace vqc {

template <int V>
struct IC {
  static constexpr int value = V;
};

// A thread's 2^R amplitudes as plain scalars (real and imaginary parts in
// separate arrays so every access has a constant index and stays in VGPRs).
template <int R>
struct St {
  static constexpr int N = 1 << R;
  float r[N];
  float i[N];
};

// Calls f(IC<p>) for a runtime register position p < R.
template <int R, typename F>
__device__ __forceinline__ void by_reg(int p, F&& f) {
  switch (p) {
    case 0: f(IC<0>{}); break;
    case 1: if constexpr (R > 1) f(IC<1>{}); break;
    case 2: if constexpr (R > 2) f(IC<2>{}); break;
    case 3: if constexpr (R > 3) f(IC<3>{}); break;
    default: if constexpr (R > 4) f(IC<4>{}); break;
  }
}

// ------------------------------------------------------------------ gates
// R_P(t) = exp(-i t P / 2) with c = cos(t/2), s = sin(t/2); the adjoint uses -s.

template <int R, int P>
__device__ __forceinline__ void rx_reg(St<R>& a, float c, float s) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
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

template <int R, int P>
__device__ __forceinline__ void ry_reg(St<R>& a, float c, float s) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
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
template <int R, int P>
__device__ __forceinline__ void rz_reg(St<R>& a, float c, float s) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float ss = (u & (1 << P)) ? s : -s;
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = c * xr - ss * xi;
    a.i[u] = c * xi + ss * xr;
  }
}

// multiply every amplitude by (c + i ss)
template <int R>
__device__ __forceinline__ void phase_all(St<R>& a, float c, float ss) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = c * xr - ss * xi;
    a.i[u] = c * xi + ss * xr;
  }
}

// CNOT with control and target on register bits: a register permutation
template <int R, int C, int T>
__device__ __forceinline__ void cnot_rr(St<R>& a) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (!(u & (1 << C)) || (u & (1 << T))) continue;
    const int v = u | (1 << T);
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = a.r[v];
    a.i[u] = a.i[v];
    a.r[v] = xr;
    a.i[v] = xi;
  }
}

// CNOT with the control on a thread / tile bit (flag) and the target on register bit T
template <int R, int T>
__device__ __forceinline__ void cnot_tr(St<R>& a, bool flag) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (u & (1 << T)) continue;
    const int v = u | (1 << T);
    const float xr = a.r[u], xi = a.i[u], yr = a.r[v], yi = a.i[v];
    a.r[u] = flag ? yr : xr;
    a.i[u] = flag ? yi : xi;
    a.r[v] = flag ? xr : yr;
    a.i[v] = flag ? xi : yi;
  }
}

// register indices u with bit p set, as a mask over u
template <int R>
__device__ __forceinline__ uint32_t reg_pattern(int p) {
  constexpr uint32_t full = R == 5 ? 0xFFFFFFFFu : ((1u << (1 << R)) - 1u);
  const uint32_t pat = p == 0 ? 0xAAAAAAAAu : p == 1 ? 0xCCCCCCCCu : p == 2 ? 0xF0F0F0F0u
                       : p == 3 ? 0xFF00FF00u : 0xFFFF0000u;
  return pat & full;
}

// tb: the bits of the amplitude position above the register bits (thread index
// within the tile, then the tile index of a streamed sample)
template <int R>
__device__ __forceinline__ uint32_t bit_mask(int p, uint32_t tb) {
  if (p < R) return reg_pattern<R>(p);
  return ((tb >> (p - R)) & 1u) ? 0xFFFFFFFFu : 0u;
}

// amplitudes whose register index u has bit u of `m` set are negated
template <int R>
__device__ __forceinline__ void negate_mask(St<R>& a, uint32_t m) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float sg = ((m >> u) & 1u) ? -1.f : 1.f;
    a.r[u] *= sg;
    a.i[u] *= sg;
  }
}

// x with its sign flipped when m == 0x80000000 (m == 0: unchanged)
__device__ __forceinline__ float flip_sign(float x, uint32_t m) {
  return __uint_as_float(__float_as_uint(x) ^ m);
}

// CZ between register positions P and Q
template <int R, int P, int Q>
__device__ __forceinline__ void cz_rr(St<R>& a) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u)
    if ((u >> P) & (u >> Q) & 1) {
      a.r[u] = -a.r[u];
      a.i[u] = -a.i[u];
    }
}

// CZ between register position P and a thread / tile bit of value `bit`
template <int R, int P>
__device__ __forceinline__ void cz_tr(St<R>& a, uint32_t bit) {
  const uint32_t m = bit << 31;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u)
    if ((u >> P) & 1) {
      a.r[u] = flip_sign(a.r[u], m);
      a.i[u] = flip_sign(a.i[u], m);
    }
}

// every amplitude negated when bit == 1 (CZ between two thread / tile bits)
template <int R>
__device__ __forceinline__ void negate_if(St<R>& a, uint32_t bit) {
  const uint32_t m = bit << 31;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    a.r[u] = flip_sign(a.r[u], m);
    a.i[u] = flip_sign(a.i[u], m);
  }
}

template <int R>
__device__ __forceinline__ void apply_rx(St<R>& a, int p, float c, float s) {
  by_reg<R>(p, [&](auto P) { rx_reg<R, decltype(P)::value>(a, c, s); });
}

template <int R>
__device__ __forceinline__ void apply_ry(St<R>& a, int p, float c, float s) {
  by_reg<R>(p, [&](auto P) { ry_reg<R, decltype(P)::value>(a, c, s); });
}

// RZ on physical bit p: register bit, or a thread / tile bit (uniform phase)
template <int R>
__device__ __forceinline__ void apply_rz(St<R>& a, int p, float c, float s, uint32_t tb) {
  if (p >= R) {
    phase_all<R>(a, c, ((tb >> (p - R)) & 1u) ? s : -s);
    return;
  }
  by_reg<R>(p, [&](auto P) { rz_reg<R, decltype(P)::value>(a, c, s); });
}

template <int R>
__device__ __forceinline__ void apply_cnot(St<R>& a, int pc, int pt, uint32_t tb) {
  if (pc >= R) {
    const bool f = (tb >> (pc - R)) & 1u;
    by_reg<R>(pt, [&](auto T) { cnot_tr<R, decltype(T)::value>(a, f); });
    return;
  }
  by_reg<R>(pc, [&](auto C) {
    by_reg<R>(pt, [&](auto T) {
      if constexpr (decltype(C)::value != decltype(T)::value)
        cnot_rr<R, decltype(C)::value, decltype(T)::value>(a);
    });
  });
}

// ------------------------------------------- fused adjoint rotation steps
// One pass over the amplitude pairs: accumulate dL/dtheta = Im <l| P |a> and
// un-apply R_P(theta) (i.e. apply R_P(-theta)) to both a and l.  Working pair by
// pair keeps only the pair's old values alive.
// Im(conj(l) a) = l.r a.i - l.i a.r ; Re(conj(l) a) = l.r a.r + l.i a.i

template <int R, int P>
__device__ __forceinline__ float adj_rx(St<R>& a, St<R>& l, float c, float s) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float ar = a.r[u], ai = a.i[u], br = a.r[v], bi = a.i[v];
    const float lr = l.r[u], li = l.i[u], mr = l.r[v], mi = l.i[v];
    // X: <l|X|a> = conj(l0) a1 + conj(l1) a0
    acc = fmaf(lr, bi, acc);
    acc = fmaf(-li, br, acc);
    acc = fmaf(mr, ai, acc);
    acc = fmaf(-mi, ar, acc);
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

template <int R, int P>
__device__ __forceinline__ float adj_ry(St<R>& a, St<R>& l, float c, float s) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float ar = a.r[u], ai = a.i[u], br = a.r[v], bi = a.i[v];
    const float lr = l.r[u], li = l.i[u], mr = l.r[v], mi = l.i[v];
    // Y a = (-i a1, i a0): Im<l|Y|a> = -Re(conj(l0) a1) + Re(conj(l1) a0)
    acc = fmaf(-lr, br, acc);
    acc = fmaf(-li, bi, acc);
    acc = fmaf(mr, ar, acc);
    acc = fmaf(mi, ai, acc);
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
template <int R, int P>
__device__ __forceinline__ float adj_rz(St<R>& a, St<R>& l, float c, float s) {
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float ar = a.r[u], ai = a.i[u], lr = l.r[u], li = l.i[u];
    float& z = (u & (1 << P)) ? a1 : a0;
    z = fmaf(lr, ai, z);
    z = fmaf(-li, ar, z);
    const float ss = (u & (1 << P)) ? -s : s;  // the inverse phase
    a.r[u] = c * ar - ss * ai;
    a.i[u] = c * ai + ss * ar;
    l.r[u] = c * lr - ss * li;
    l.i[u] = c * li + ss * lr;
  }
  return a0 - a1;
}

// RZ on a thread / tile bit: the Z sign and the inverse phase are uniform
template <int R>
__device__ __forceinline__ float adj_rz_uniform(St<R>& a, St<R>& l, float c, float s, bool one) {
  float acc = 0.f;
  const float ss = one ? -s : s;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float ar = a.r[u], ai = a.i[u], lr = l.r[u], li = l.i[u];
    acc = fmaf(lr, ai, acc);
    acc = fmaf(-li, ar, acc);
    a.r[u] = c * ar - ss * ai;
    a.i[u] = c * ai + ss * ar;
    l.r[u] = c * lr - ss * li;
    l.i[u] = c * li + ss * lr;
  }
  return one ? -acc : acc;
}

// ------------------------------------------------ tangent form (generated kernels)
// R_P(theta) is written as R_P(2 phi') P^m (up to a global phase) with
// phi' = theta/2 - m pi/2 in [-pi/4, pi/4], and R_P(2 phi') = cos(phi') (I - i t P)
// with t = tan(phi').  The generated kernels apply only I - i t P, one FMA per
// real component, keep the per-sample factors cos(phi') aside (applied in blocks
// by rescale) and carry the Paulis P^m as a frame that only flips signs of t,
// of <Z_q> and of gradients (tables built per sample before the schedule).

// (I - i t X) on the pair (u, u + 2^P)
template <int R, int P>
__device__ __forceinline__ void rx_t(St<R>& a, float t) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float xr = a.r[u], xi = a.i[u], yr = a.r[v], yi = a.i[v];
    a.r[u] = fmaf(t, yi, xr);
    a.i[u] = fmaf(-t, yr, xi);
    a.r[v] = fmaf(t, xi, yr);
    a.i[v] = fmaf(-t, xr, yi);
  }
}

// (I - i t Y) = [1, -t; t, 1]
template <int R, int P>
__device__ __forceinline__ void ry_t(St<R>& a, float t) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float xr = a.r[u], xi = a.i[u], yr = a.r[v], yi = a.i[v];
    a.r[u] = fmaf(-t, yr, xr);
    a.i[u] = fmaf(-t, yi, xi);
    a.r[v] = fmaf(t, xr, yr);
    a.i[v] = fmaf(t, xi, yi);
  }
}

// (I - i t Z) on register bit P: amplitude times (1 - i t z), z = +-1
template <int R, int P>
__device__ __forceinline__ void rz_t(St<R>& a, float t) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float tz = (u & (1 << P)) ? -t : t;
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = fmaf(tz, xi, xr);
    a.i[u] = fmaf(-tz, xr, xi);
  }
}

// every amplitude times (1 - i tz) (RZ on a thread / tile bit, tz = t z)
template <int R>
__device__ __forceinline__ void phase_t(St<R>& a, float tz) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float xr = a.r[u], xi = a.i[u];
    a.r[u] = fmaf(tz, xi, xr);
    a.i[u] = fmaf(-tz, xr, xi);
  }
}

template <int R>
__device__ __forceinline__ void rescale(St<R>& a, float f) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    a.r[u] *= f;
    a.i[u] *= f;
  }
}

// Adjoint steps: Im<l| P |a> at the gate's output, then (I + i t P) on both.
template <int R, int P>
__device__ __forceinline__ float adj_rx_t(St<R>& a, St<R>& l, float t) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float ar = a.r[u], ai = a.i[u], br = a.r[v], bi = a.i[v];
    const float lr = l.r[u], li = l.i[u], mr = l.r[v], mi = l.i[v];
    acc = fmaf(lr, bi, acc);
    acc = fmaf(-li, br, acc);
    acc = fmaf(mr, ai, acc);
    acc = fmaf(-mi, ar, acc);
    a.r[u] = fmaf(-t, bi, ar);
    a.i[u] = fmaf(t, br, ai);
    a.r[v] = fmaf(-t, ai, br);
    a.i[v] = fmaf(t, ar, bi);
    l.r[u] = fmaf(-t, mi, lr);
    l.i[u] = fmaf(t, mr, li);
    l.r[v] = fmaf(-t, li, mr);
    l.i[v] = fmaf(t, lr, mi);
  }
  return acc;
}

template <int R, int P>
__device__ __forceinline__ float adj_ry_t(St<R>& a, St<R>& l, float t) {
  float acc = 0.f;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (u & (1 << P)) continue;
    const int v = u | (1 << P);
    const float ar = a.r[u], ai = a.i[u], br = a.r[v], bi = a.i[v];
    const float lr = l.r[u], li = l.i[u], mr = l.r[v], mi = l.i[v];
    acc = fmaf(-lr, br, acc);
    acc = fmaf(-li, bi, acc);
    acc = fmaf(mr, ar, acc);
    acc = fmaf(mi, ai, acc);
    a.r[u] = fmaf(t, br, ar);
    a.i[u] = fmaf(t, bi, ai);
    a.r[v] = fmaf(-t, ar, br);
    a.i[v] = fmaf(-t, ai, bi);
    l.r[u] = fmaf(t, mr, lr);
    l.i[u] = fmaf(t, mi, li);
    l.r[v] = fmaf(-t, lr, mr);
    l.i[v] = fmaf(-t, li, mi);
  }
  return acc;
}

template <int R, int P>
__device__ __forceinline__ float adj_rz_t(St<R>& a, St<R>& l, float t) {
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float ar = a.r[u], ai = a.i[u], lr = l.r[u], li = l.i[u];
    float& z = (u & (1 << P)) ? a1 : a0;
    z = fmaf(lr, ai, z);
    z = fmaf(-li, ar, z);
    const float tz = (u & (1 << P)) ? t : -t;  // the inverse: (1 + i t z)
    a.r[u] = fmaf(tz, ai, ar);
    a.i[u] = fmaf(-tz, ar, ai);
    l.r[u] = fmaf(tz, li, lr);
    l.i[u] = fmaf(-tz, lr, li);
  }
  return a0 - a1;
}

// RZ on a thread / tile bit of value `one`: uniform z
template <int R>
__device__ __forceinline__ float adj_phase_t(St<R>& a, St<R>& l, float t, uint32_t one) {
  float acc = 0.f;
  const float tz = one ? t : -t;  // the inverse phase (1 + i t z)
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float ar = a.r[u], ai = a.i[u], lr = l.r[u], li = l.i[u];
    acc = fmaf(lr, ai, acc);
    acc = fmaf(-li, ar, acc);
    a.r[u] = fmaf(tz, ai, ar);
    a.i[u] = fmaf(-tz, ar, ai);
    l.r[u] = fmaf(tz, li, lr);
    l.i[u] = fmaf(-tz, lr, li);
  }
  return one ? -acc : acc;
}

template <int R>
__device__ __forceinline__ float adjoint_rotation(int op, St<R>& a, St<R>& l, int p, float c,
                                                  float s, uint32_t tb) {
  float g = 0.f;
  if (op == OP_RX) {
    by_reg<R>(p, [&](auto P) { g = adj_rx<R, decltype(P)::value>(a, l, c, s); });
  } else if (op == OP_RY) {
    by_reg<R>(p, [&](auto P) { g = adj_ry<R, decltype(P)::value>(a, l, c, s); });
  } else if (p >= R) {
    g = adj_rz_uniform<R>(a, l, c, s, (tb >> (p - R)) & 1u);
  } else {
    by_reg<R>(p, [&](auto P) { g = adj_rz<R, decltype(P)::value>(a, l, c, s); });
  }
  return g;
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

// A copy of x that the compiler cannot prove equal to x.  Addresses formed
// from it are recomputed instead of being kept alive (and spilled) across the
// whole schedule.
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

// butterfly sum over `width` consecutive lanes (power of two <= 64); every lane
// of the segment ends with the same, order-fixed value.  The empty asm keeps
// the shuffles where all lanes are active (see group_sum).
__device__ __forceinline__ float seg_sum(float v, int width) {
  asm volatile("" : "+v"(v));
  for (int m = 1; m < width; m <<= 1) v += __shfl_xor(v, m, 64);
  asm volatile("" : "+v"(v));
  return v;
}

// the same over the whole wave, fully unrolled
__device__ __forceinline__ float wave_sum(float v) {
  asm volatile("" : "+v"(v));
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m, 64);
  asm volatile("" : "+v"(v));
  return v;
}

// v from another lane through a DPP lane pattern (every lane reads a valid lane)
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// The value lane (lane ^ 2^J) of the wave holds, for J < 4: lanes 1, 2 and 8
// apart are one DPP move (quad_perm 1032, quad_perm 2301, row_ror 8), 4 apart
// two (row_half_mirror, then quad_perm 3210: (i ^ 7) ^ 3 = i ^ 4).  Every lane
// is a valid source, so no old value is needed.
template <int CTRL>
__device__ __forceinline__ float mov_dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
template <int J>
__device__ __forceinline__ float xlane(float v) {
  static_assert(J >= 0 && J < 4, "lane bit");
  if constexpr (J == 0) return mov_dpp_f<0xB1>(v);
  else if constexpr (J == 1) return mov_dpp_f<0x4E>(v);
  else if constexpr (J == 2) return mov_dpp_f<0x1B>(mov_dpp_f<0x141>(v));
  else return mov_dpp_f<0x128>(v);
}

// Exchange of register bit RB with lane bit J without LDS: the qubit on
// register bit RB moves to lane bit J and back.  The amplitude at register u,
// lane L stays where bit RB of u equals bit J of L, and otherwise comes from
// lane L ^ 2^J, register u ^ 2^RB.  For J = 4 and 5 this is exactly what
// gfx950's permlane16 / permlane32 swaps do to the pair (a[u0], a[u1]): the
// odd 16-lane rows (upper 32 lanes) of the first operand trade places with the
// even rows (lower 32 lanes) of the second.  Below that, a DPP move and a
// select per value.
// x where the mask is set, y elsewhere
__device__ __forceinline__ float bit_select(uint32_t m, float x, float y) {
  return __uint_as_float((__float_as_uint(x) & m) | (__float_as_uint(y) & ~m));
}

__device__ __forceinline__ void swap_pair16(float& x0, float& x1) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x0), __float_as_uint(x1), false,
                                                  false);
  x0 = __uint_as_float(r[0]);
  x1 = __uint_as_float(r[1]);
}
__device__ __forceinline__ void swap_pair32(float& x0, float& x1) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x0), __float_as_uint(x1), false,
                                                  false);
  x0 = __uint_as_float(r[0]);
  x1 = __uint_as_float(r[1]);
}

template <int R, int RB, int J>
__device__ __forceinline__ void lane_swap(St<R>& a, uint32_t lane) {
#pragma unroll
  for (int u0 = 0; u0 < St<R>::N; ++u0) {
    if (u0 & (1 << RB)) continue;
    const int u1 = u0 | (1 << RB);
    if constexpr (J == 4) {
      swap_pair16(a.r[u0], a.r[u1]);
      swap_pair16(a.i[u0], a.i[u1]);
    } else if constexpr (J == 5) {
      swap_pair32(a.r[u0], a.r[u1]);
      swap_pair32(a.i[u0], a.i[u1]);
    } else {
      // a bit-select (one bitfield insert per value): written as a select the
      // compiler turns the four choices into a divergent branch
      const uint32_t m = 0u - ((lane >> J) & 1u);
      const float r0 = xlane<J>(a.r[u1]), i0 = xlane<J>(a.i[u1]);
      const float r1 = xlane<J>(a.r[u0]), i1 = xlane<J>(a.i[u0]);
      a.r[u0] = bit_select(m, r0, a.r[u0]);
      a.i[u0] = bit_select(m, i0, a.i[u0]);
      a.r[u1] = bit_select(m, a.r[u1], r1);
      a.i[u1] = bit_select(m, a.i[u1], i1);
    }
  }
}

// ------------------------------------------------------- gates on lane bits
// With 4 amplitudes per thread and every other qubit on a lane bit of the
// sample, the generated kernels apply RX, RY and CNOT targets on lane bit J
// directly: the partner amplitude of a pair sits in lane ^ 2^J, same register,
// and is read with xlane<J> (DPP).  `hi` is the thread's lane bit J.

// RX(theta): both sides of the pair take c a - i s a_partner
// (the moved value is the first factor of a plain product, so the DPP move
// folds into the multiply)
template <int R, int J>
__device__ __forceinline__ void rx_lane(St<R>& a, float c, float s) {
  const float ns = -s;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float tr = xlane<J>(a.i[u]) * s, ti = xlane<J>(a.r[u]) * ns;
    a.r[u] = fmaf(c, a.r[u], tr);
    a.i[u] = fmaf(c, a.i[u], ti);
  }
}

// RY(theta) = [c, -s; s, c]: the side with the bit clear takes c a - s a_partner,
// the side with it set c a + s a_partner
template <int R, int J>
__device__ __forceinline__ void ry_lane(St<R>& a, float c, float s, uint32_t hi) {
  const float sl = flip_sign(s, (hi ^ 1u) << 31);
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float tr = xlane<J>(a.r[u]) * sl, ti = xlane<J>(a.i[u]) * sl;
    a.r[u] = fmaf(c, a.r[u], tr);
    a.i[u] = fmaf(c, a.i[u], ti);
  }
}

// Adjoint RX on lane bit J: this lane's share of Im<l|X|a>, then RX(-theta) on
// both states (c a + i s a_partner).  The share pairs this lane's a with the
// partner's l (the pair's two terms are split between its lanes either way);
// the partner's l is needed for the update too, the partner's a only once, in
// a product the DPP move folds into.
template <int R, int J>
__device__ __forceinline__ float adj_rx_lane(St<R>& a, St<R>& l, float c, float s) {
  float acc = 0.f;
  const float ns = -s;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float qr = xlane<J>(l.r[u]), qi = xlane<J>(l.i[u]);
    const float ar = a.r[u], ai = a.i[u];
    acc = fmaf(qr, ai, acc);
    acc = fmaf(-qi, ar, acc);
    const float tr = xlane<J>(ai) * ns, ti = xlane<J>(ar) * s;
    a.r[u] = fmaf(c, ar, tr);
    a.i[u] = fmaf(c, ai, ti);
    l.r[u] = fmaf(c, l.r[u], qi * ns);
    l.i[u] = fmaf(c, l.i[u], qr * s);
  }
  return acc;
}

// Adjoint RY on lane bit J: Im<l|Y|a> over a pair is
// Re(conj(l1) a0) - Re(conj(l0) a1); the side with the bit clear holds a0 and
// takes +Re(conj(l_partner) a), the other side -.  RY(-theta) = [c, s; -s, c]
template <int R, int J>
__device__ __forceinline__ float adj_ry_lane(St<R>& a, St<R>& l, float c, float s, uint32_t hi) {
  float acc = 0.f;
  const float sl = flip_sign(s, hi << 31);
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float qr = xlane<J>(l.r[u]), qi = xlane<J>(l.i[u]);
    const float ar = a.r[u], ai = a.i[u];
    acc = fmaf(qr, ar, acc);
    acc = fmaf(qi, ai, acc);
    const float tr = xlane<J>(ar) * sl, ti = xlane<J>(ai) * sl;
    a.r[u] = fmaf(c, ar, tr);
    a.i[u] = fmaf(c, ai, ti);
    l.r[u] = fmaf(c, l.r[u], qr * sl);
    l.i[u] = fmaf(c, l.i[u], qi * sl);
  }
  return hi ? -acc : acc;
}

// The tangent form (I -+ i t P, see rx_t) on lane bit J: one FMA per real
// component, the partner's value moved by DPP.
// (I - i t X): a.r + t b.i, a.i - t b.r with b the partner amplitude
template <int R, int J>
__device__ __forceinline__ void rx_lane_t(St<R>& a, float t) {
  const float nt = -t;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float br = xlane<J>(a.r[u]), bi = xlane<J>(a.i[u]);
    a.r[u] = fmaf(t, bi, a.r[u]);
    a.i[u] = fmaf(nt, br, a.i[u]);
  }
}

// (I - i t Y) = [1, -t; t, 1]: the partner enters with -t on the side with
// the bit clear and +t on the other
template <int R, int J>
__device__ __forceinline__ void ry_lane_t(St<R>& a, float t, uint32_t hi) {
  const float tl = flip_sign(t, (hi ^ 1u) << 31);
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float br = xlane<J>(a.r[u]), bi = xlane<J>(a.i[u]);
    a.r[u] = fmaf(tl, br, a.r[u]);
    a.i[u] = fmaf(tl, bi, a.i[u]);
  }
}

// Adjoint steps on lane bit J: this lane's share of Im<l|P|a> (as in
// adj_rx_lane / adj_ry_lane), then the inverse (I + i t P) on both states.
template <int R, int J>
__device__ __forceinline__ float adj_rx_lane_t(St<R>& a, St<R>& l, float t) {
  float acc = 0.f;
  const float nt = -t;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float qr = xlane<J>(l.r[u]), qi = xlane<J>(l.i[u]);
    const float br = xlane<J>(a.r[u]), bi = xlane<J>(a.i[u]);
    const float ar = a.r[u], ai = a.i[u];
    acc = fmaf(qr, ai, acc);
    acc = fmaf(-qi, ar, acc);
    a.r[u] = fmaf(nt, bi, ar);
    a.i[u] = fmaf(t, br, ai);
    l.r[u] = fmaf(nt, qi, l.r[u]);
    l.i[u] = fmaf(t, qr, l.i[u]);
  }
  return acc;
}

template <int R, int J>
__device__ __forceinline__ float adj_ry_lane_t(St<R>& a, St<R>& l, float t, uint32_t hi) {
  float acc = 0.f;
  const float tl = flip_sign(t, hi << 31);  // +t with the bit clear, -t with it set
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const float qr = xlane<J>(l.r[u]), qi = xlane<J>(l.i[u]);
    const float br = xlane<J>(a.r[u]), bi = xlane<J>(a.i[u]);
    const float ar = a.r[u], ai = a.i[u];
    acc = fmaf(qr, ar, acc);
    acc = fmaf(qi, ai, acc);
    a.r[u] = fmaf(tl, br, ar);
    a.i[u] = fmaf(tl, bi, ai);
    l.r[u] = fmaf(tl, qr, l.r[u]);
    l.i[u] = fmaf(tl, qi, l.i[u]);
  }
  return hi ? -acc : acc;
}

// CNOT with the target on lane bit J and the control on register bit C: the
// amplitudes with the control set trade places with the partner lane's
template <int R, int C, int J>
__device__ __forceinline__ void cnot_rl(St<R>& a) {
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    if (!(u & (1 << C))) continue;
    a.r[u] = xlane<J>(a.r[u]);
    a.i[u] = xlane<J>(a.i[u]);
  }
}

// CNOT with the target on lane bit J and the control on a thread / tile bit
// (the same in both lanes of a pair)
template <int R, int J>
__device__ __forceinline__ void cnot_tl(St<R>& a, uint32_t flag) {
  const uint32_t m = 0u - flag;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    a.r[u] = bit_select(m, xlane<J>(a.r[u]), a.r[u]);
    a.i[u] = bit_select(m, xlane<J>(a.i[u]), a.i[u]);
  }
}

// CNOT with the target on lane bit J and the control on lane bit C >= 2: the
// lanes with the control set are whole DPP banks (C = 2, 3: lane bits 2 and 3
// within a row) or rows (C = 4, 5), so one DPP move under that mask gives them
// the partner's value while the others keep their own (no select).
template <int J, int ROW, int BANK>
__device__ __forceinline__ float masked_xlane(float v) {
  static_assert(J >= 0 && J < 4, "lane bit");
  const int x = __float_as_int(v);
  if constexpr (J == 0)
    return __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0xB1, ROW, BANK, false));
  else if constexpr (J == 1)
    return __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x4E, ROW, BANK, false));
  else if constexpr (J == 2)
    return __int_as_float(__builtin_amdgcn_update_dpp(
        x, __float_as_int(mov_dpp_f<0x141>(v)), 0x1B, ROW, BANK, false));
  else
    return __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x128, ROW, BANK, false));
}

template <int R, int J, int C>
__device__ __forceinline__ void cnot_ll(St<R>& a) {
  static_assert(C >= 2 && C <= 5 && C != J, "control on a bank or row bit");
  constexpr int BANK = C == 2 ? 0xA : C == 3 ? 0xC : 0xF;
  constexpr int ROW = C == 4 ? 0xA : C == 5 ? 0xC : 0xF;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    a.r[u] = masked_xlane<J, ROW, BANK>(a.r[u]);
    a.i[u] = masked_xlane<J, ROW, BANK>(a.i[u]);
  }
}

// Sum over aligned groups of W lanes (W a power of two <= 64).  Every lane of a
// group ends with the group's sum; the pairing order is fixed, so the result is
// deterministic.  Pairs, quads, 8- and 16-lane rows use DPP (quad_perm 1032 and
// 2301, row_half_mirror, row_mirror), 32 lanes a swizzle (xor 16), 64 lanes the
// four row sums read as scalars.
template <int W>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(W >= 1 && W <= 64 && (W & (W - 1)) == 0, "group width");
  // The empty asm statements pin the cross-lane steps to this point of the
  // program: without them the compiler may sink the whole sum into a branch
  // taken by one lane only (the lane that consumes it), where the lanes it reads
  // from are inactive.
  asm volatile("" : "+v"(v));
  if (W >= 2) v += dpp_f<0xB1>(v);
  if (W >= 4) v += dpp_f<0x4E>(v);
  if (W >= 8) v += dpp_f<0x141>(v);
  if (W >= 16) v += dpp_f<0x140>(v);
  if (W == 32) v += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x401F));
  if (W == 64) {
    const int x = __float_as_int(v);
    v = (__int_as_float(__builtin_amdgcn_readlane(x, 0)) +
         __int_as_float(__builtin_amdgcn_readlane(x, 16))) +
        (__int_as_float(__builtin_amdgcn_readlane(x, 32)) +
         __int_as_float(__builtin_amdgcn_readlane(x, 48)));
  }
  asm volatile("" : "+v"(v));
  return v;
}

// XOR of the columns selected by the bits of u (u < 2^R)
template <int R>
__device__ __forceinline__ uint32_t xor_cols(int u, const uint32_t (&c)[R]) {
  uint32_t o = 0;
#pragma unroll
  for (int b = 0; b < R; ++b)
    if (u & (1 << b)) o ^= c[b];
  return o;
}

// LDS exchange: write the amplitudes at lam(old index), read lam(new index).
// col[0..k) are the write-side columns, col[k..2k) the read-side columns.  The
// buffer is planar (real parts, then imaginary parts, `plane` floats apart) so
// every access is a 32-bit one: no 64-bit register tuples enter the schedule
// loop, and 32 lanes hit 32 banks.  Addresses are formed in bytes (columns
// scaled by 4 once), so an access costs one XOR and no shift.

// The thread's byte offsets of its write and read slots (register bits 0).
template <int R>
__device__ __forceinline__ void exchange_bases(const uint32_t* col, int k, int t, int stid, int sl,
                                               uint32_t& bw, uint32_t& br) {
  // an opaque thread index: the addresses of one exchange are not merged with
  // equal ones of later exchanges (which would keep them alive in between)
  const uint32_t ot = opaque((uint32_t)stid);
  bw = 0;
  br = 0;
#pragma unroll
  for (int i = 0; i < kMaxTileQubits - 2; ++i) {
    if (i < t && ((ot >> i) & 1)) {
      bw ^= col[R + i];
      br ^= col[k + R + i];
    }
  }
  // samples sharing a 32-lane group are spread over different banks
  const uint32_t lowmask = (1u << (k < kBankBits ? k : kBankBits)) - 1u;
  const uint32_t xs = ((uint32_t)sl << t) & lowmask;
  const uint32_t base = (uint32_t)sl << k;
  bw = (base | (bw ^ xs)) << 2;
  br = (base | (br ^ xs)) << 2;
}

template <int R>
__device__ __forceinline__ void exchange_at(St<R>& a, float* xbuf, uint32_t plane,
                                            const uint32_t* col, int k, uint32_t bw,
                                            uint32_t br) {
  uint32_t cw[R], cr[R];
#pragma unroll
  for (int b = 0; b < R; ++b) {
    cw[b] = col[b] << 2;
    cr[b] = col[k + b] << 2;
  }
  unsigned char* xr = reinterpret_cast<unsigned char*>(xbuf);
  unsigned char* xi = xr + 4 * plane;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const uint32_t o = bw ^ xor_cols<R>(u, cw);
    *reinterpret_cast<float*>(xr + o) = a.r[u];
    *reinterpret_cast<float*>(xi + o) = a.i[u];
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const uint32_t o = br ^ xor_cols<R>(u, cr);
    a.r[u] = *reinterpret_cast<const float*>(xr + o);
    a.i[u] = *reinterpret_cast<const float*>(xi + o);
  }
  __syncthreads();
}

// fo: byte offset XORed into every write address, which resolves a swap frame
// (register index u holds position u ^ f: its slot is that of u, XOR the
// columns of f's bits)
template <int R>
__device__ __forceinline__ void exchange(St<R>& a, float* xbuf, uint32_t plane,
                                         const uint32_t* col, int k, int t, int stid, int sl,
                                         uint32_t fo = 0u) {
  uint32_t bw, br;
  exchange_bases<R>(col, k, t, stid, sl, bw, br);
  exchange_at<R>(a, xbuf, plane, col, k, bw ^ fo, br);
}

// The same permutation of two states (the adjoint's psi and lambda), one after
// the other through the buffer, with the slot bases formed once.
template <int R>
__device__ __forceinline__ void exchange2(St<R>& a, St<R>& l, float* xbuf, uint32_t plane,
                                          const uint32_t* col, int k, int t, int stid, int sl,
                                          uint32_t fo = 0u) {
  uint32_t bw, br;
  exchange_bases<R>(col, k, t, stid, sl, bw, br);
  exchange_at<R>(a, xbuf, plane, col, k, bw ^ fo, br);
  exchange_at<R>(l, xbuf, plane, col, k, bw ^ fo, br);
}

// ------------------------------------------------------------ swap frame
// In the generated kernels (tangent form) a CNOT whose control sits on a
// thread / tile bit c and whose target sits on register bit r does not move
// data: the thread records that its registers along bit r are swapped iff c
// is set (a frame F = X_r^c, kept as a sign mask fs_r = c << 31), and the
// state held is F times the true one.  A later gate G then runs as F G F:
// RY and RZ on bit r with the angle negated (X RY X = RY(-theta), likewise
// RZ), RX and everything on other bits unchanged, a register CNOT from r to
// r' adds the frame X_r' (F CNOT = CNOT F X_r'); the adjoint's gradient of a
// negated rotation is negated (Im <lambda| X P X |psi> = -Im <lambda|P|psi>
// for P = Y, Z).  The frame is resolved where the positions matter: folded
// into the write addresses of an LDS exchange (register u goes to position
// u ^ f; the addresses are XOR-linear in u), or, before anything else that
// reads positions (lane swaps, CZs, epilogues, stores), by one conditional
// swap per frame bit.

// ------------------------------------------------------- schedule runner

// Context of one workgroup's walk through an instruction stream.
// One angle occurrence: its source (parameter / input / constant) and index,
// and (mul, add), or (cos, sin)(theta/2) when the angle is constant.
struct OccRec {
  int32_t src, idx;
  float a, b;
};

struct Walk {
  const uint32_t* cols;
  float* xbuf;        // planar exchange buffer: plane floats of real parts, then imaginary
  uint32_t plane;
  const float2* tab;  // (cos, sin)(theta/2), [occurrence][S]
  const float* ma;    // (mul, add) per occurrence, or null: gradients carry mul
  float* acc;         // gradient accumulators [slot][G]
  int k, t, S, G;
  int stid, sl, grp, width;
  uint32_t tb;        // tile bits above the register bits
  bool leader;
  bool never;         // false, but not provably so (see gate_boundary)
  unsigned char* smem;  // the workgroup's LDS (tables of the generated kernels)
};

// Ends the current basic block with a uniform branch that is never taken.  The
// generated kernels put one after every rotation, so that instruction
// selection and scheduling work gate by gate: one block for a whole circuit
// makes them keep values alive across it (and compile slowly).
__device__ __forceinline__ void gate_boundary(const Walk& w) {
  if (w.never) asm volatile("");
}

// Angle table of a one-sample workgroup held in registers: lane j of the
// wave's copy row m holds occurrence 64 m + j, read at a gate into scalar
// registers.  The values are uniform over the wave, so a gate needs no LDS
// read (whose latency a lone wave per SIMD cannot hide).
__device__ __forceinline__ float2 table_row(const Walk& w, int m, int last) {
  const int j = 64 * m + (int)__lane_id();
  return w.tab[j < last ? j : last];
}

template <int J>
__device__ __forceinline__ float2 table_entry(const float2 row) {
  return make_float2(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(row.x), J)),
                     __int_as_float(__builtin_amdgcn_readlane(__float_as_int(row.y), J)));
}

// the same for a table of floats (the adjoint's gradient signs)
__device__ __forceinline__ float table_row(const float* tab, int m, int last) {
  const int j = 64 * m + (int)__lane_id();
  return tab[j < last ? j : last];
}

template <int J>
__device__ __forceinline__ float table_entry(const float row) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(row), J));
}

// Bit p >= R of the amplitude position (a thread or tile bit).  Taken from an
// opaque copy of tb so that the compiler recomputes it at each gate instead of
// keeping every bit (and the masks built from it) alive across the schedule.
template <int R>
__device__ __forceinline__ uint32_t tile_bit(const Walk& w, int p) {
  return (opaque(w.tb) >> (p - R)) & 1u;
}

// Adds a rotation's gradient partial (summed over the lanes of a sample) to
// the sample's accumulator row of this wave.  One writer per address keeps the
// order of additions fixed.
template <bool WIDE>
__device__ __forceinline__ void acc_add(const Walk& w, int slot, float g) {
  g = WIDE ? wave_sum(g) : seg_sum(g, w.width);
  if (w.leader) atomicAdd(&w.acc[slot * w.G + w.grp], g);
}

// Runs `n_ins` instructions on psi (a) and, for the adjoint, lambda (l).
// WIDE: every sample spans whole waves (the reduction width is 64).
template <int R, bool BWD, bool WIDE>
__device__ __forceinline__ void run_schedule(St<R>& a, St<R>& l, const uint32_t* ins, int n_ins,
                                             const Walk& w) {
  for (int pc = 0; pc < n_ins; ++pc) {
    const uint32_t w0 = ins[2 * pc];
    const uint32_t arg = ins[2 * pc + 1];
    const int op = w0 & 31;
    const int pa = (w0 >> 5) & 31;
    const int pb = (w0 >> 10) & 31;
    if (op == OP_EXCHANGE) {
      if (BWD)
        exchange2<R>(a, l, w.xbuf, w.plane, w.cols + arg, w.k, w.t, w.stid, w.sl);
      else
        exchange<R>(a, w.xbuf, w.plane, w.cols + arg, w.k, w.t, w.stid, w.sl);
      continue;
    }
    if (op == OP_CNOT) {
      apply_cnot<R>(a, pa, pb, w.tb);
      if (BWD) apply_cnot<R>(l, pa, pb, w.tb);
      continue;
    }
    if (op == OP_CZ) {
      const uint32_t m = bit_mask<R>(pa, w.tb) & bit_mask<R>(pb, w.tb);
      negate_mask<R>(a, m);
      if (BWD) negate_mask<R>(l, m);
      continue;
    }
    const float2 cs = w.tab[arg * w.S + w.sl];
    if (!BWD) {
      if (op == OP_RX) apply_rx<R>(a, pa, cs.x, cs.y);
      else if (op == OP_RY) apply_ry<R>(a, pa, cs.x, cs.y);
      else apply_rz<R>(a, pa, cs.x, cs.y, w.tb);
    } else {
      // dL/dtheta = Im <lambda| P |psi>, then psi, lambda <- R(-theta) psi, lambda
      const float g = adjoint_rotation<R>(op, a, l, pa, cs.x, cs.y, w.tb);
      const int slot = (int)(w0 >> 16) - 1;
      if (slot >= 0) acc_add<WIDE>(w, slot, w.ma ? g * w.ma[2 * arg] : g);
    }
  }
}

// Parameter resolution: (cos, sin)(theta/2) for every occurrence and sample of
// the workgroup, theta = mul * value + add (occ_ma, or the value itself when
// occ_ma is null).  Constant angles come precomputed from the compile phase.
// fd_slots > 0 (central differences): sample bb of the launch is the shifted
// copy r = bb mod (2 fd_slots) of input row bb / (2 fd_slots), in which slot
// fd_base + r / 2 (parameters, then inputs) is moved by +fd_h (r even) or
// -fd_h.  Sched::occ gives an occurrence's source, index and (mul, add), or
// its (cos, sin) when constant: read from the plan's arrays, or compiled in.
template <typename Sched>
__device__ __forceinline__ void angle_table(float2* tab, int n_occ, int S, int64_t b0, int64_t B,
                                            const int32_t* occ_src, const int32_t* occ_idx,
                                            const float* occ_cs, const float* occ_ma,
                                            const float* params, int P,
                                            const float* inputs, int F, int tid, int nthreads,
                                            int n_params = 0, int fd_slots = 0,
                                            float fd_h = 0.f, int fd_base = 0) {
  if (Sched::kNocc >= 0) {  // compiled-in sizes: constant trip counts
    n_occ = Sched::kNocc;
    S = Sched::kS;
  }
  const int total = n_occ * S;
  // Four rounds at a time: the rounds' occurrence records, then their values,
  // are loaded together, so that a chunk waits for two load latencies before
  // its sincos.  The value loads are unconditional (a lane with nothing to
  // read reads the first word of occ_src, a 256-byte aligned region of the
  // schedule that other regions follow), and the empty asm keeps the compiler
  // from sinking them into the branches that use them.
  constexpr int kRounds = 4;
#pragma unroll
  for (int c0 = 0; c0 < total; c0 += kRounds * nthreads) {
    OccRec oc[kRounds];
    float th[kRounds], shift[kRounds];
    bool var[kRounds];
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const int i = c0 + r * nthreads + tid;
      oc[r] = Sched::occ(occ_src, occ_idx, occ_cs, occ_ma, i < total ? i / S : 0);
    }
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const int i = c0 + r * nthreads + tid;
      const bool live = i < total;
      const int64_t bb = b0 + (live ? i % S : 0);
      var[r] = live && oc[r].src != kSrcConst && bb < B;
      int64_t row = bb;
      shift[r] = 0.f;
      if (fd_slots > 0) {
        const int64_t per = 2 * (int64_t)fd_slots;
        row = bb / per;
        const int rr = (int)(bb - row * per);
        const int slot = oc[r].src == kSrcParam ? oc[r].idx : n_params + oc[r].idx;
        if (slot == fd_base + (rr >> 1)) shift[r] = (rr & 1) ? -fd_h : fd_h;
      }
      const float* src = !var[r] ? reinterpret_cast<const float*>(occ_src)
                         : oc[r].src == kSrcParam ? params + row * P + oc[r].idx
                                                  : inputs + row * F + oc[r].idx;
      th[r] = *src;
    }
#pragma unroll
    for (int r = 0; r < kRounds; ++r) asm volatile("" : "+v"(th[r]));
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const int i = c0 + r * nthreads + tid;
      if (i >= total) continue;
      float c = 1.f, sn = 0.f;  // rows past the batch
      if (oc[r].src == kSrcConst) {
        c = oc[r].a;
        sn = oc[r].b;
      } else if (var[r]) {
        float t = th[r] + shift[r];
        if (occ_ma) t = fmaf(oc[r].a, t, oc[r].b);
        sincosf(0.5f * t, &sn, &c);
      }
      tab[i] = make_float2(c, sn);
    }
  }
}

// lambda = H psi with H = sum_q g_q Z(q), where Z(q) is the Z-string measured for
// qubit q's <Z> (Z_q itself, or Z_q pulled back through the circuit's trailing
// entanglers); Sched::zmask gives its physical bits under `phys`.
template <int R, typename Sched>
__device__ __forceinline__ void make_lambda(St<R>& l, const St<R>& a, const float* g, int n,
                                            const uint8_t* phys, const uint32_t* zm, uint32_t tb,
                                            bool valid, const float* esign = nullptr) {
  constexpr uint32_t rbits = (1u << R) - 1u;
  float h[St<R>::N];
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) h[u] = 0.f;
  if (valid) {
#pragma unroll
    for (int q = 0; q < (Sched::kN >= 0 ? Sched::kN : n); ++q) {
      float gq = esign ? g[q] * esign[q] : g[q];
      const uint32_t pm = Sched::zmask(phys, zm, q);
      if (__builtin_popcount(tb & (pm >> R)) & 1) gq = -gq;
#pragma unroll
      for (int u = 0; u < St<R>::N; ++u)
        h[u] += (__builtin_popcount((uint32_t)u & pm & rbits) & 1) ? -gq : gq;
    }
  }
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    l.r[u] = h[u] * a.r[u];
    l.i[u] = h[u] * a.i[u];
  }
}

// Signed probability sums of this workgroup's amplitudes for every measured
// qubit q: ez[q * G + grp] = sum over the group's amplitudes of
// (-1)^{parity(x & Z(q))} |a|^2, Z(q) the qubit's measured Z-string.  Must be
// called by every thread; ez may alias the exchange buffer.
template <int R, typename Sched>
__device__ __forceinline__ void z_partials(const St<R>& a, float* ez, int n, const uint8_t* phys,
                                           const uint32_t* zm, const Walk& w) {
  constexpr uint32_t rbits = (1u << R) - 1u;
  float pj[St<R>::N];
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) pj[u] = a.r[u] * a.r[u] + a.i[u] * a.i[u];
  __syncthreads();  // the exchange buffer may still be read by other threads
#pragma unroll
  for (int q = 0; q < (Sched::kN >= 0 ? Sched::kN : n); ++q) {
    const uint32_t pm = Sched::zmask(phys, zm, q);
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < St<R>::N; ++u)
      v += (__builtin_popcount((uint32_t)u & pm & rbits) & 1) ? -pj[u] : pj[u];
    if (__builtin_popcount(w.tb & (pm >> R)) & 1) v = -v;
    v = Sched::lane_sum(v, w);
    if (const float* es = Sched::esigns(w)) v *= es[q];
    if (w.leader) ez[q * w.G + w.grp] = v;
  }
  __syncthreads();
}

// The precompiled kernels' schedule runner: interprets the instruction stream;
// the circuit's constants come from the plan's arrays in device memory.
struct InterpSched {
  // number of qubits when fixed at compile time, else -1 (then A.n)
  static constexpr int kN = -1;
  // occurrences and samples per workgroup when fixed at compile time, else -1
  static constexpr int kNocc = -1, kS = -1;
  // the streaming passes compute their tables (no per-sample table kernel)
  static constexpr bool kLoadTables = false;
  // a pass's flags other than PF_INIT when fixed at compile time, else -1
  static constexpr int kFixedFlags = -1;
  // the training step's product head (generated passes only): the first
  // forward pass starts from the product state, the last adjoint pass writes
  // the head partials
  static constexpr bool kProductStart = false, kHeadPartials = false;
  // physical bits of qubit q's measured Z-string under the mapping the epilogue /
  // lambda use (zm: the logical strings, or null for Z_q itself)
  __device__ __forceinline__ static uint32_t zmask(const uint8_t* phys, const uint32_t* zm,
                                                   int q) {
    if (!zm) return 1u << phys[q];
    uint32_t m = zm[q], pm = 0u;
    while (m) {
      pm |= 1u << phys[__builtin_ctz(m)];
      m &= m - 1u;
    }
    return pm;
  }
  __device__ __forceinline__ static OccRec occ(const int32_t* src, const int32_t* idx,
                                               const float* cs, const float* ma, int o) {
    OccRec r;
    r.src = src[o];
    r.idx = idx[o];
    if (r.src == kSrcConst) {
      r.a = cs[2 * o];
      r.b = cs[2 * o + 1];
    } else if (ma) {
      r.a = ma[2 * o];
      r.b = ma[2 * o + 1];
    } else {
      r.a = 1.f;
      r.b = 0.f;
    }
    return r;
  }
  template <int R, bool BWD, bool WIDE>
  __device__ __forceinline__ static void run(St<R>& a, St<R>& l, const Walk& w,
                                             const uint32_t* ins, int n_ins) {
    run_schedule<R, BWD, WIDE>(a, l, ins, n_ins, w);
  }
  // sum over the lanes of one sample within the wave
  __device__ __forceinline__ static float lane_sum(float v, const Walk& w) {
    return seg_sum(v, w.width);
  }
  // per-sample tables built before the schedule (none here), and the
  // constants they need, read at the start of the kernel (none)
  struct Pre {};
  __device__ __forceinline__ static Pre preload(int) { return Pre(); }
  __device__ __forceinline__ static void prepare(const Walk&, int, int, const Pre&) {}
  // signs of <Z_q> of the thread's sample (none: the state is the true state)
  __device__ __forceinline__ static const float* esigns(const Walk&) { return nullptr; }
};

// Cotangent g_j = dL/dE_j of one sample's row e[0..n) for the loss heads of the
// C ABI (y: the sample's target, B: the batch the mean runs over).
__device__ __forceinline__ float loss_cot(int kind, const float* e, float y, int n, int j,
                                          int64_t B) {
  if (kind == kLossSum) return 1.f;
  if (kind == kLossMean) return 1.f / (float)n;
  if (kind == kLossMseZ0) return j == 0 ? 2.f * (e[0] - y) / (float)B : 0.f;
  float s = 0.f;
  for (int q = 0; q < n; ++q) s += e[q];
  s /= (float)n;
  return 2.f * (s - y) / ((float)n * (float)B);
}

// ------------------------------------------------------ resident body

// One launch for a tile of S samples (T = 2^t threads each); Sched runs the
// instruction stream (the interpreter of the precompiled kernels, or the
// straight-line code generated for one circuit).

template <int WG, int R>
__device__ __forceinline__ Walk resident_walk(const TileArgs& A, unsigned char* smem) {
  Walk w;
  const int tid = threadIdx.x;
  const int T = 1 << A.t;
  w.cols = A.cols;
  w.xbuf = reinterpret_cast<float*>(smem);
  w.plane = (uint32_t)WG << R;
  w.tab = reinterpret_cast<float2*>(smem + A.lds_tab);
  w.ma = A.occ_ma;
  w.acc = reinterpret_cast<float*>(smem + A.lds_acc);
  w.k = A.k;
  w.t = A.t;
  w.S = A.S;
  w.G = A.G;
  w.stid = tid & (T - 1);
  w.sl = tid >> A.t;
  w.width = T < 64 ? T : 64;
  w.grp = T < 64 ? w.sl : (tid >> 6);
  w.leader = (tid & (w.width - 1)) == 0;
  w.never = A.B < 0;
  w.smem = smem;
  w.tb = (uint32_t)w.stid;
  return w;
}

// <Z_q> of the workgroup's samples from the ez partials: e[s * n + q] (when e
// is not null) and expvals rows.  Every thread must call it.
__device__ __forceinline__ void resident_expvals(const TileArgs& A, const float* ez, float* e,
                                                 int WG) {
  const int S = A.S;
  const int64_t b0 = (int64_t)blockIdx.x * S;
  for (int i = threadIdx.x; i < A.n * S; i += WG) {
    const int q = i / S;
    const int s = i - q * S;
    const int64_t bb = b0 + s;
    float v;
    if (A.t >= 6) {
      v = 0.f;
      for (int g = 0; g < A.G; ++g) v += ez[q * A.G + g];
    } else {
      v = ez[q * A.G + s];
    }
    if (e) e[s * A.n + q] = v;
    if (bb < A.B && A.expvals) A.expvals[bb * A.n + q] = v;
  }
}

// dparams / dinputs rows from the per-group accumulators (after a barrier).
__device__ __forceinline__ void resident_grads(const TileArgs& A, const float* acc, int WG) {
  const int S = A.S;
  const int64_t b0 = (int64_t)blockIdx.x * S;
  for (int i = threadIdx.x; i < A.n_slots * S; i += WG) {
    const int slot = i / S;
    const int s = i - slot * S;
    const int64_t bb = b0 + s;
    if (bb >= A.B) continue;
    float v;
    if (A.t >= 6) {
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

// Logical basis index of a thread's amplitudes under a mapping phys[q] (logical
// qubit -> physical bit): x(u) = xt ^ (XOR of rq[b] over the set bits b of u).
// Qubits n..k-1 pad small circuits to the tile; amplitudes with a padding bit
// set (thread bits: pt, register bits: pr) are identically zero.
template <int R>
struct LogicalIndex {
  uint32_t xt, pr, rq[R];
  bool pt;
  __device__ __forceinline__ uint32_t at(int u) const {
    uint32_t x = xt;
#pragma unroll
    for (int b = 0; b < R; ++b)
      if (u & (1 << b)) x ^= rq[b];
    return x;
  }
};

// The logical index of each of the thread's amplitudes under mapping `phys`,
// as the XOR of per-qubit columns: 1 << q, or pc[q] where the index is mapped
// through the trailing entanglers' basis permutation (probabilities).
template <int R>
__device__ __forceinline__ LogicalIndex<R> logical_index(const uint8_t* phys, int n, int k,
                                                         uint32_t tb,
                                                         const uint32_t* pc = nullptr) {
  LogicalIndex<R> li;
  li.xt = 0u;
  li.pr = 0u;
  li.pt = false;
#pragma unroll
  for (int b = 0; b < R; ++b) li.rq[b] = 0u;
  for (int q = 0; q < k; ++q) {
    const int p = phys[q];
    const uint32_t col = q < n ? (pc ? pc[q] : 1u << q) : 0u;
    if (p >= R) {
      const uint32_t bit = (tb >> (p - R)) & 1u;
      if (q < n) li.xt ^= bit ? col : 0u;
      else li.pt = li.pt || bit;
    } else {
#pragma unroll
      for (int b = 0; b < R; ++b)
        if (p == b) {
          if (q < n) li.rq[b] = col;
          else li.pr |= 1u << b;
        }
    }
  }
  return li;
}

// X part of the Pauli frame the tangent form leaves on the state: bit q is set
// where the frame anticommutes with Z_q (its <Z_q> sign is -1).  Basis state
// x of the register state is basis state x ^ mask of the true state.
__device__ __forceinline__ uint32_t frame_xmask(const float* es, int n) {
  uint32_t m = 0u;
  if (es)
    for (int q = 0; q < n; ++q)
      if (es[q] < 0.f) m |= 1u << q;
  return m;
}

// Resident forward from the caller's initial states (Algorithm 1, optional
// Psi_0): the workgroup's rows are staged in LDS with coalesced loads, then
// every thread picks its amplitudes by logical index under the start mapping.
template <int WG, int R>
__device__ __forceinline__ void load_initial(St<R>& a, const TileArgs& A, const Walk& w) {
  const int N = 1 << A.n;
  const int64_t b0 = (int64_t)blockIdx.x * A.S;
  const int64_t have = (A.B - b0) * N;  // amplitudes of the workgroup's real samples
  float* re = w.xbuf;
  float* im = w.xbuf + A.S * N;
  const float2* src = reinterpret_cast<const float2*>(A.psi0) + b0 * N;
  for (int i = threadIdx.x; i < A.S * N; i += WG) {
    const float2 v = i < have ? src[i] : make_float2(0.f, 0.f);
    re[i] = v.x;
    im[i] = v.y;
  }
  __syncthreads();
  const LogicalIndex<R> li = logical_index<R>(A.start_phys, A.n, A.k, w.tb);
  const int row = w.sl * N;
#pragma unroll
  for (int u = 0; u < St<R>::N; ++u) {
    const bool live = !li.pt && !(u & li.pr);
    const uint32_t x = li.at(u);
    a.r[u] = live ? re[row + x] : 0.f;
    a.i[u] = live ? im[row + x] : 0.f;
  }
  __syncthreads();  // the exchange buffer is reused by the sweep
}

// Basis-state probabilities of the workgroup's final states (Sec. 3: the other
// output of the execute phase), permuted to logical order through LDS and
// written with coalesced stores.  Every thread must call it.
template <int WG, int R, typename Sched>
__device__ __forceinline__ void resident_probs(const St<R>& a, const TileArgs& A, const Walk& w) {
  const int N = 1 << A.n;
  const uint32_t xm = frame_xmask(Sched::esigns(w), A.n);
  const LogicalIndex<R> li = logical_index<R>(A.end_phys, A.n, A.k, w.tb, A.pcol);
  float* pb = w.xbuf;
  __syncthreads();  // the exchange buffer may still be read
  if (!li.pt) {
    const int row = w.sl * N;
#pragma unroll
    for (int u = 0; u < St<R>::N; ++u)
      if (!(u & li.pr)) pb[row + (li.at(u) ^ xm)] = a.r[u] * a.r[u] + a.i[u] * a.i[u];
  }
  __syncthreads();
  const int64_t b0 = (int64_t)blockIdx.x * A.S;
  const int64_t have = (A.B - b0) * N;
  float* dst = A.probs + b0 * N;
  for (int i = threadIdx.x; i < A.S * N; i += WG)
    if (i < have) dst[i] = pb[i];
}

template <int R>
__device__ __forceinline__ void zero_state(St<R>& a, int stid) {
#pragma unroll
  for (int j = 0; j < St<R>::N; ++j) {
    a.r[j] = 0.f;
    a.i[j] = 0.f;
  }
  if (stid == 0) a.r[0] = 1.f;
}

template <int WG, bool BWD, int R, typename Sched>
__device__ __forceinline__ void resident_body(const TileArgs& A, unsigned char* smem) {
  constexpr int NA = 1 << R;
  const int tid = threadIdx.x;
  const Walk w = resident_walk<WG, R>(A, smem);
  const int64_t b0 = (int64_t)blockIdx.x * A.S;
  const int64_t b = b0 + w.sl;
  const bool valid = b < A.B;

  const typename Sched::Pre pre = Sched::preload(tid);
  angle_table<Sched>(reinterpret_cast<float2*>(smem + A.lds_tab), A.n_occ, A.S, b0, A.B,
                     A.occ_src, A.occ_idx, A.occ_cs, A.occ_ma, A.params, A.pstride, A.inputs,
                     A.F, tid, WG, A.P, A.fd_slots, A.fd_h);
  if (BWD)
    for (int i = tid; i < A.n_slots * A.G; i += WG) w.acc[i] = 0.f;
  __syncthreads();
  Sched::prepare(w, tid, WG, pre);

  St<R> a, l;
  if (!BWD) {
    if (A.psi0) load_initial<WG, R>(a, A, w);
    else zero_state<R>(a, w.stid);
  } else {
    const float2* ws = reinterpret_cast<const float2*>(A.ws);
    float2 v[NA];
#pragma unroll
    for (int j = 0; j < NA; ++j) v[j] = ws[((size_t)blockIdx.x * NA + j) * WG + tid];
#pragma unroll
    for (int j = 0; j < NA; ++j) split(v[j], a.r[j], a.i[j]);
    make_lambda<R, Sched>(l, a, A.grad_out + (valid ? b : 0) * A.n, A.n, A.end_phys, A.zmask,
                          w.tb, valid, Sched::esigns(w));
  }

  Sched::template run<R, BWD, (WG > 64)>(a, l, w, A.ins, A.n_ins);

  if (!BWD) {
    if (A.ws) {
      float2* ws = reinterpret_cast<float2*>(A.ws);
#pragma unroll
      for (int j = 0; j < NA; ++j)
        ws[((size_t)blockIdx.x * NA + j) * WG + tid] = make_float2(a.r[j], a.i[j]);
    }
    z_partials<R, Sched>(a, w.xbuf, A.n, A.end_phys, A.zmask, w);
    resident_expvals(A, w.xbuf, nullptr, WG);
    if (A.probs) resident_probs<WG, R, Sched>(a, A, w);
  } else {
    __syncthreads();
    resident_grads(A, w.acc, WG);
  }
}

// Training step in one launch: forward (FS), <Z>, the loss head's cotangent,
// lambda = (sum_j g_j Z_j) psi and the adjoint sweep (BS).  The state stays on
// chip between the two sweeps; nothing is saved to HBM.
// ------------------------------------------------------------ product head
// A qubit's head is the run of rotations on it before any entangler touches
// it.  Heads commute with every other gate up to their ends, so the state after
// all of them is the product of one-qubit states phi_q = U_q |0> applied to
// |0...0> (Sec. 3's initial state).  The generated training step builds that
// product instead of running the head rotations, and its adjoint stops where
// the heads end.  There, with psi the product state, the gradient of a head
// rotation R_P of qubit q, Im <lambda|P|psi> at its place, equals
// Im <mu|P|phi> in the qubit's own two dimensions: phi the qubit's state after
// the rotation, mu = (I_q (x) <phi_{not q}|) lambda walked back through the
// rotations of the head after it.  The 2-vectors v_q = (I_q (x) <phi_{not q}|)
// lambda are sums over the whole state; one lane per qubit then walks its head.

// Lane q's head (q < n), one entry per step i: word = occurrence | kind << 16
// (kind 0 X, 1 Y, 2 Z, 3 no step), gradient slot + 1 (0: a constant angle),
// chain-rule factor of the angle.
template <int L>
struct HeadPre {
  uint32_t w[L];
  int32_t s[L];
  float m[L];
};

// No head (the default of the step kernel).
struct NoHead {
  static constexpr bool kOn = false;
  struct Pre {};
  __device__ __forceinline__ static Pre preload(int) { return Pre(); }
};

// One head step in LDS: the qubit's state after it, and its record.
struct HeadRec {
  float4 phi;  // (a.re, a.im, b.re, b.im) of a|0> + b|1>
  uint32_t word;
  int32_t slot1;
  float mul;
  float pad;
};

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}
// conj(a) * b
__device__ __forceinline__ float2 cmulc(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, a.y * b.y), fmaf(a.x, b.y, -a.y * b.x));
}
__device__ __forceinline__ float2 cadd(float2 a, float2 b) {
  return make_float2(a.x + b.x, a.y + b.y);
}

// P (a|0> + b|1>) for P = X (kind 0), Y (1), Z (2)
__device__ __forceinline__ void pauli2(uint32_t kind, float2 a, float2 b, float2& pa, float2& pb) {
  pa = kind == 0u ? b : kind == 1u ? make_float2(b.y, -b.x) : a;
  pb = kind == 0u ? a : kind == 1u ? make_float2(-a.y, a.x) : make_float2(-b.x, -b.y);
}

__device__ __forceinline__ float lane_value(float v, int q) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), q));
}

// Reduce-scatter of 16 values over the wave's 64 lanes: lane L returns the sum
// of value L % 16 over all lanes.  Value-index bit b pairs with lane bit b: bit
// 2 first (row_half_mirror pairs lane l with l ^ 7 while every lane still holds
// all 16 values), then bits 0 and 1 (quad_perm 1032, 2301) and 3 (row_ror 8);
// two more additions (lane ^ 16 by a swizzle, lane ^ 32) complete the sums.
// The pairing order is fixed, so the sums are deterministic.  Written with
// named values: selects between elements of one array would become a
// run-time index into it.
#define VQC_RS_PAIR(CTRL, HB, K, A, B) \
  do {                                 \
    const float k_ = (HB) ? (B) : (A); \
    const float s_ = (HB) ? (A) : (B); \
    K = k_ + dpp_f<CTRL>(s_);          \
  } while (0)
__device__ __forceinline__ float wave_reduce16(const float (&v)[16], uint32_t lane) {
  float x0 = v[0], x1 = v[1], x2 = v[2], x3 = v[3], x4 = v[4], x5 = v[5], x6 = v[6], x7 = v[7];
  float x8 = v[8], x9 = v[9], x10 = v[10], x11 = v[11], x12 = v[12], x13 = v[13], x14 = v[14],
        x15 = v[15];
  const bool h2 = (lane >> 2) & 1u, h0 = lane & 1u, h1 = (lane >> 1) & 1u, h3 = (lane >> 3) & 1u;
  float y0, y1, y2, y3, y4, y5, y6, y7;  // value bit 2 gone: y[q] holds values with bits 0, 1, 3 of q
  VQC_RS_PAIR(0x141, h2, y0, x0, x4);
  VQC_RS_PAIR(0x141, h2, y1, x1, x5);
  VQC_RS_PAIR(0x141, h2, y2, x2, x6);
  VQC_RS_PAIR(0x141, h2, y3, x3, x7);
  VQC_RS_PAIR(0x141, h2, y4, x8, x12);
  VQC_RS_PAIR(0x141, h2, y5, x9, x13);
  VQC_RS_PAIR(0x141, h2, y6, x10, x14);
  VQC_RS_PAIR(0x141, h2, y7, x11, x15);
  float z0, z1, z2, z3;  // value bit 0 gone
  VQC_RS_PAIR(0xB1, h0, z0, y0, y1);
  VQC_RS_PAIR(0xB1, h0, z1, y2, y3);
  VQC_RS_PAIR(0xB1, h0, z2, y4, y5);
  VQC_RS_PAIR(0xB1, h0, z3, y6, y7);
  float w0, w1;  // value bit 1 gone
  VQC_RS_PAIR(0x4E, h1, w0, z0, z1);
  VQC_RS_PAIR(0x4E, h1, w1, z2, z3);
  float tot;  // value bit 3 gone
  VQC_RS_PAIR(0x128, h3, tot, w0, w1);
  tot += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(tot), 0x401F));
  tot += __shfl_xor(tot, 32, 64);
  return tot;
}
#undef VQC_RS_PAIR

// One head step on the qubit's state: (c I - i s P) phi, (c, s) the rotation's
// exact (cos, sin)(theta / 2) (kind 3: no step).
__device__ __forceinline__ void head_step(const Walk& w, uint32_t word, float2& fa, float2& fb) {
  const uint32_t kind = word >> 16;
  float2 cs = w.tab[word & 0xFFFFu];
  if (kind == 3u) cs = make_float2(1.f, 0.f);
  float2 pa, pb;
  pauli2(kind, fa, fb, pa, pb);
  fa = make_float2(fmaf(cs.x, fa.x, cs.y * pa.y), fmaf(cs.x, fa.y, -cs.y * pa.x));
  fb = make_float2(fmaf(cs.x, fb.x, cs.y * pb.y), fmaf(cs.x, fb.y, -cs.y * pb.x));
}

// Lane q's head state phi_q (lanes of every wave; lanes >= n walk a clamped
// copy whose values are not used).
template <int L>
__device__ __forceinline__ void head_state(const Walk& w, const HeadPre<L>& hp, float2& fa,
                                           float2& fb) {
  fa = make_float2(1.f, 0.f);
  fb = make_float2(0.f, 0.f);
#pragma unroll
  for (int i = 0; i < L; ++i) head_step(w, hp.w[i], fa, fb);
}

// Lane q's walk through the head of qubit q (lanes of every wave do it; wave
// 0 records each step's state in LDS): fa, fb end as the qubit's state.
template <int L>
__device__ __forceinline__ void head_walk(const Walk& w, const HeadPre<L>& hp, HeadRec* rec,
                                          float4* fin, int n, float2& fa, float2& fb) {
  const int lane = (int)__lane_id();
  const bool writer = lane < n && threadIdx.x < 64;
  fa = make_float2(1.f, 0.f);
  fb = make_float2(0.f, 0.f);
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const uint32_t word = hp.w[i];
    head_step(w, word, fa, fb);
    if (writer) {
      HeadRec r;
      r.phi = make_float4(fa.x, fa.y, fb.x, fb.y);
      r.word = word;
      r.slot1 = hp.s[i];
      r.mul = hp.m[i];
      r.pad = 0.f;
      rec[lane * L + i] = r;
    }
  }
  if (writer) fin[lane] = make_float4(fa.x, fa.y, fb.x, fb.y);
}

// Lane q's walk back through its head from mu = v_q = (m0, m1): at every step
// (last first) the rotation's gradient Im <mu|P|phi>, phi the recorded state
// after it, goes to emit(i, record, gradient); then mu <- (c I + i s P) mu.
template <int L, typename Emit>
__device__ __forceinline__ void head_back(const Walk& w, const HeadRec* rec, int q, float2 m0,
                                          float2 m1, Emit&& emit) {
#pragma unroll
  for (int i = L - 1; i >= 0; --i) {
    const HeadRec r = rec[q * L + i];
    const uint32_t kind = r.word >> 16;
    if (kind == 3u) continue;
    const float2 cs = w.tab[r.word & 0xFFFFu];
    float2 p0, p1;
    pauli2(kind, make_float2(r.phi.x, r.phi.y), make_float2(r.phi.z, r.phi.w), p0, p1);
    // Im(conj(mu_0) (P phi)_0 + conj(mu_1) (P phi)_1)
    const float g = fmaf(m0.x, p0.y, -m0.y * p0.x) + fmaf(m1.x, p1.y, -m1.y * p1.x);
    emit(i, r, g);
    float2 q0, q1;
    pauli2(kind, m0, m1, q0, q1);
    m0 = make_float2(fmaf(cs.x, m0.x, -cs.y * q0.y), fmaf(cs.x, m0.y, cs.y * q0.x));
    m1 = make_float2(fmaf(cs.x, m1.x, -cs.y * q1.y), fmaf(cs.x, m1.y, cs.y * q1.x));
  }
}

// Sums of the per-thread values v[0 .. NV) over the workgroup (each wave by
// wave_reduce16, then the waves through the exchange buffer, in a fixed
// order): thread j < NV gets sum j.  Every thread calls it; it starts with a
// barrier (the exchange buffer may still be in use) and ends with one.
template <int WG, int NV>
__device__ __forceinline__ float workgroup_sums(const float (&v)[NV], float* red) {
  const uint32_t lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  __syncthreads();
#pragma unroll
  for (int c = 0; c < NV / 16; ++c) {
    float x16[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) x16[j] = v[16 * c + j];
    const float tot = wave_reduce16(x16, lane);
    if (lane < 16u) red[wave * NV + 16 * c + (int)lane] = tot;
  }
  __syncthreads();
  float s = 0.f;
  if ((int)threadIdx.x < NV)
    for (int g = 0; g < WG / 64; ++g) s += red[g * NV + threadIdx.x];
  __syncthreads();
  return s;
}

// The head gradients from the per-thread 2-vector partials v[4 q .. 4 q + 3]
// (v_q(0), v_q(1) as re, im): sums over the workgroup (each wave, then the
// waves through the exchange buffer), then lane q of wave 0 walks qubit q's
// head back and adds each rotation's gradient to accumulator group 0.  Every
// thread calls it, after a barrier.
template <int WG, int L, int NV>
__device__ __forceinline__ void head_finish(const float (&v)[NV], const Walk& w,
                                            const HeadRec* rec, int n) {
  const uint32_t lane = __lane_id();
  const int wave = threadIdx.x >> 6;
  float* red = w.xbuf;
#pragma unroll
  for (int c = 0; c < NV / 16; ++c) {
    float x16[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) x16[j] = v[16 * c + j];
    const float tot = wave_reduce16(x16, lane);
    if (lane < 16u) red[wave * NV + 16 * c + (int)lane] = tot;
  }
  __syncthreads();
  const int q = threadIdx.x;
  if (q >= n) return;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int g = 0; g < WG / 64; ++g) {
    s.x += red[g * NV + 4 * q];
    s.y += red[g * NV + 4 * q + 1];
    s.z += red[g * NV + 4 * q + 2];
    s.w += red[g * NV + 4 * q + 3];
  }
  head_back<L>(w, rec, q, make_float2(s.x, s.y), make_float2(s.z, s.w),
               [&](int, const HeadRec& r, float g) {
                 if (r.slot1 > 0) atomicAdd(&w.acc[(r.slot1 - 1) * w.G], g * r.mul);
               });
}

// The streaming training step's head gradients and gradient rows: one
// workgroup of WG threads per sample, after its last adjoint pass.  Every
// slot's sum over the sample's tiles' partials (in tile order) is loaded
// first, so that those loads overlap the rest.  v_q is the sum of the tiles'
// head partials (in tile order); lane q walks qubit q's head forward
// (recording the states) and back, and each rotation's gradient times its
// chain-rule factor goes to an LDS row of slots: written in place when no two
// head rotations share a slot, else summed per slot over a fixed list of
// terms (H::add_grads).  Each slot's value is its tile sum plus that row,
// written to dparams / dinputs.
template <int WG, typename H>
__device__ __forceinline__ void head_finish_stream(const PassArgs& A, unsigned char* smem) {
  constexpr int L = H::kL, NV = H::kNV, N = H::kN, NS = H::kNS, T = 1 << H::kNG;
  constexpr int PT = (NS + WG - 1) / WG;  // slots per thread
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.x;
  const int64_t row0 = b << H::kNG;
  const float* gp = A.gpart + row0 * NS;
  // a compile-time tile count: every load of a sum is in flight at once
  float tsum[PT];
#pragma unroll
  for (int k = 0; k < PT; ++k) {
    const int s = tid + k * WG;
    float v = 0.f;
    if (s < NS) {
#pragma unroll
      for (int g = 0; g < T; ++g) v += gp[g * NS + s];
    }
    tsum[k] = v;
  }
  Walk w;
  w.tab = reinterpret_cast<const float2*>(A.tabs) + b * A.n_occ;  // exact (cos, sin) of heads
  HeadRec* rec = reinterpret_cast<HeadRec*>(smem);
  float4* fin = reinterpret_cast<float4*>(smem + N * L * 32);
  float* vs = reinterpret_cast<float*>(smem + N * L * 32 + N * 16);
  float* gs = vs + NV;     // [n][L]
  float* hs = gs + N * L;  // [NS]
  const HeadPre<L> hp = H::head_pre(tid);
  float2 fa, fb;
  head_walk<L>(w, hp, rec, fin, N, fa, fb);
  for (int j = tid; j < NV; j += WG) {
    float s = 0.f;
#pragma unroll
    for (int g = 0; g < T; ++g) s += A.vpart[(row0 + g) * NV + j];
    vs[j] = s;
  }
  for (int j = tid; j < NS; j += WG) hs[j] = 0.f;
  __syncthreads();
  if (tid < N)
    head_back<L>(w, rec, tid, make_float2(vs[4 * tid], vs[4 * tid + 1]),
                 make_float2(vs[4 * tid + 2], vs[4 * tid + 3]),
                 [&](int i, const HeadRec& r, float g) {
                   if constexpr (H::kUniqueSlots) {
                     if (r.slot1 > 0) hs[r.slot1 - 1] = g * r.mul;
                   } else {
                     gs[tid * L + i] = g * r.mul;
                   }
                 });
  __syncthreads();
  if constexpr (!H::kUniqueSlots) {
    H::add_grads(gs, hs, tid, WG);
    __syncthreads();
  }
#pragma unroll
  for (int k = 0; k < PT; ++k) {
    const int s = tid + k * WG;
    if (s >= NS) break;
    const float v = tsum[k] + hs[s];
    if (s < A.P) {
      if (A.dparams) A.dparams[b * A.P + s] = v;
    } else if (A.dinputs) {
      A.dinputs[b * A.F + (s - A.P)] = v;
    }
  }
}

template <int WG, int R, typename FS, typename BS, typename HD = NoHead>
__device__ __forceinline__ void resident_step_body(const TileArgs& A, unsigned char* smem) {
  const int tid = threadIdx.x;
  const Walk w = resident_walk<WG, R>(A, smem);
  const int64_t b0 = (int64_t)blockIdx.x * A.S;
  const bool valid = b0 + w.sl < A.B;
  float* e = reinterpret_cast<float*>(smem + A.lds_e);  // [S][n]
  float* g = e + A.S * A.n;                             // [S][n]
  float* ys = g + A.S * A.n;                            // [S] the loss head's targets

  // The loss head's targets and the frame tables' constants are read first, so
  // that their latency is hidden.  The target load is unconditional, so that
  // no branch makes the kernel wait for it at once; without targets it reads
  // occ_src (a 256-byte aligned region of the schedule that other regions
  // follow, so always readable).
  const int64_t yrow = b0 + (tid < A.S ? tid : 0);
  const float* yp = A.target ? A.target + (yrow < A.B ? yrow : A.B - 1)
                             : reinterpret_cast<const float*>(A.occ_src);
  const float y0 = *yp;
  const typename FS::Pre pre = FS::preload(tid);
  const typename HD::Pre hpre = HD::preload(tid);
  angle_table<FS>(reinterpret_cast<float2*>(smem + A.lds_tab), A.n_occ, A.S, b0, A.B,
                  A.occ_src, A.occ_idx, A.occ_cs, A.occ_ma, A.params, A.pstride, A.inputs, A.F,
                  tid, WG);
  // stored where the table's loads have completed anyway (a load in the loss
  // loop would wait for the stores of E issued before it)
  if (tid < A.S) ys[tid] = A.target && b0 + tid < A.B ? y0 : 0.f;
  for (int i = tid; i < A.n_slots * A.G; i += WG) w.acc[i] = 0.f;
  __syncthreads();
  FS::prepare(w, tid, WG, pre);  // the tables of both sweeps

  St<R> a, l;
  if constexpr (HD::kOn)
    HD::template init<R>(a, w, hpre);
  else
    zero_state<R>(a, w.stid);
  FS::template run<R, false, (WG > 64)>(a, l, w, A.ins, A.n_ins);
  z_partials<R, FS>(a, w.xbuf, A.n, A.end_phys, A.zmask, w);
  resident_expvals(A, w.xbuf, e, WG);
  __syncthreads();
  for (int i = tid; i < A.S * A.n; i += WG) {
    const int s = i / A.n;
    const int q = i - s * A.n;
    const int64_t bb = b0 + s;
    const float y = ys[s];
    const float v = loss_cot(A.loss, e + s * A.n, y, A.n, q, A.B);
    g[i] = v;
    if (A.cot_out && bb < A.B) A.cot_out[bb * A.n + q] = v;
  }
  __syncthreads();
  make_lambda<R, FS>(l, a, g + w.sl * A.n, A.n, A.end_phys, A.zmask, w.tb, valid,
                     FS::esigns(w));
  BS::template run<R, true, (WG > 64)>(a, l, w, A.ins_b, A.n_ins_b);
  __syncthreads();
  if constexpr (HD::kOn) {
    HD::template grads<WG, R>(l, w);
    __syncthreads();
  }
  resident_grads(A, w.acc, WG);
}

// ----------------------------------------------------- streaming kernel
// One pass over B * 2^ng tiles of 2^k amplitudes (2^(k-R) threads x 2^R).
// A tile is loaded in the memory layout the pass reads and stored in the one
// it writes: tile rank r (the amplitude's position among the k local qubits
// ordered by address bit) is r = stid + 2^(k-R) j, so consecutive lanes touch
// consecutive addresses.  Addresses are the XOR of per-bit columns (io_*).

template <int R>
__device__ __forceinline__ void io_offsets(const uint32_t* io, int k, int ng, int stid, int g,
                                           uint32_t& base, uint32_t (&off)[1 << R]) {
  const int nt = k - R;
  base = 0;
#pragma unroll
  for (int i = 0; i < kMaxTileQubits - 2; ++i)
    if (i < nt && ((stid >> i) & 1)) base ^= io[i];
  for (int i = 0; i < ng; ++i)
    if ((g >> i) & 1) base ^= io[k + i];
  uint32_t c[R];
#pragma unroll
  for (int b = 0; b < R; ++b) c[b] = io[nt + b];
#pragma unroll
  for (int j = 0; j < (1 << R); ++j) off[j] = xor_cols<R>(j, c);
}

// A sample's state as a raw buffer (base: its first amplitude, `bytes` its
// size; an access beyond it reads zero and stores nothing).  The load and
// store columns are single address bits, distinct over the tile's ranks and
// global bits, so a lane's bits (base) and a register's (off, uniform over the
// workgroup) never overlap and their XOR is their sum: the lane's byte offset
// is the access's vector offset and the register's its scalar offset, with no
// address arithmetic per amplitude.
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t state_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ float2 amp_load(__amdgpu_buffer_rsrc_t r, uint32_t base_b, uint32_t off) {
  const uint32_t so = (uint32_t)__builtin_amdgcn_readfirstlane((int)(off << 3));
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, base_b, so, 0);
  return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
}

__device__ __forceinline__ void amp_store(__amdgpu_buffer_rsrc_t r, uint32_t base_b, uint32_t off,
                                          float re, float im) {
  const uint32_t so = (uint32_t)__builtin_amdgcn_readfirstlane((int)(off << 3));
  u32x2 v;
  v.x = __float_as_uint(re);
  v.y = __float_as_uint(im);
  __builtin_amdgcn_raw_buffer_store_b64(v, r, base_b, so, 0);
}

// All loads are issued before the first split, so that they overlap.
template <int R>
__device__ __forceinline__ void load_tile(St<R>& a, __amdgpu_buffer_rsrc_t src, uint32_t base,
                                          const uint32_t (&off)[1 << R]) {
  const uint32_t base_b = base << 3;
  float2 v[1 << R];
#pragma unroll
  for (int j = 0; j < (1 << R); ++j) v[j] = amp_load(src, base_b, off[j]);
#pragma unroll
  for (int j = 0; j < (1 << R); ++j) split(v[j], a.r[j], a.i[j]);
}

// The per-sample tables of the streaming passes (generated kernels, tangent
// form): one workgroup per sample computes the angle table and the frame
// signs of every occurrence (Sched::prepare over all of them) once, and
// writes (t, cos phi'), the adjoint's gradient signs and the <Z> signs for
// every pass of the call to read (so that no pass repeats the sincos, the
// divisions and the parity sums).
template <int WG, typename Sched>
__device__ __forceinline__ void table_body(const PassArgs& A, unsigned char* smem) {
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.x;
  Walk w;
  w.tab = reinterpret_cast<float2*>(smem);
  w.smem = smem;
  const typename Sched::Pre pre = Sched::preload(tid);
  angle_table<Sched>(const_cast<float2*>(w.tab), A.n_occ, 1, b, A.B, A.occ_src, A.occ_idx,
                     A.occ_cs, A.occ_ma, A.params, A.pstride, A.inputs, A.F, tid, WG, A.P,
                     A.fd_slots, A.fd_h, A.fd_base);
  __syncthreads();
  Sched::prepare(w, tid, WG, pre);  // ends with a barrier
  const float* gm = reinterpret_cast<const float*>(smem + Sched::kOffGm);
  const float* es = Sched::esigns(w);
  float2* T = reinterpret_cast<float2*>(A.tabs) + b * A.n_occ;
  float* Gs = A.gsig + b * A.n_occ;
  for (int i = tid; i < A.n_occ; i += WG) {
    T[i] = w.tab[i];
    Gs[i] = gm[i];
  }
  for (int q = tid; q < A.n; q += WG) A.esig[b * A.n + q] = es[q];
  if (A.gpart) {
    // the training step's gradient partials of this sample, cleared for its adjoint
    float* gp = A.gpart + (b << A.ng) * A.n_slots;
    for (int i = tid; i < (A.n_slots << A.ng); i += WG) gp[i] = 0.f;
  }
}

template <bool BWD, int R, int K, typename Sched>
__device__ __forceinline__ void stream_body(const PassArgs& A, unsigned char* smem) {
  static_assert(K <= kMaxTileQubits && K - R >= 6, "tile shape");
  constexpr int WG = 1 << (K - R);
  constexpr int NA = 1 << R;
  constexpr int G = WG / 64;
  float* xbuf = reinterpret_cast<float*>(smem);
  float2* tab = reinterpret_cast<float2*>(smem + A.lds_tab);
  float* acc = reinterpret_cast<float*>(smem + A.lds_acc);
  const int tid = threadIdx.x;
  const int64_t blk = blockIdx.x;
  const int64_t b = blk >> A.ng;
  const int g = (int)(blk & ((1 << A.ng) - 1));
  Walk w;
  w.cols = A.cols;
  w.xbuf = xbuf;
  w.plane = (uint32_t)WG * NA;
  w.tab = tab;
  w.ma = A.occ_ma;
  w.acc = acc;
  w.k = A.k;
  w.t = A.k - R;
  w.S = 1;
  w.G = G;
  w.stid = tid;
  w.sl = 0;
  w.width = 64;
  w.grp = tid >> 6;
  w.leader = (tid & 63) == 0;
  w.never = A.B < 0;
  w.smem = smem;
  w.tb = (uint32_t)tid | ((uint32_t)g << w.t);

  if constexpr (Sched::kLoadTables) {
    // the sample's tables, written once per call by the table kernel
    Sched::load_tables(w, A, b, tid, WG);
    if (BWD)
      for (int i = tid; i < A.n_pslots * G; i += WG) acc[i] = 0.f;
    __syncthreads();
  } else {
    const typename Sched::Pre pre = Sched::preload(tid);
    angle_table<Sched>(tab, A.n_occ, 1, b, A.B, A.occ_src, A.occ_idx, A.occ_cs, A.occ_ma,
                       A.params, A.pstride, A.inputs, A.F, tid, WG, A.P, A.fd_slots, A.fd_h,
                       A.fd_base);
    if (BWD)
      for (int i = tid; i < A.n_pslots * G; i += WG) acc[i] = 0.f;
    __syncthreads();
    Sched::prepare(w, tid, WG, pre);
  }

  // A generated pass knows its flags (all but PF_INIT, which a caller's Psi_0
  // clears): a runtime branch between forming lambda and loading it would have
  // the compiler copy the whole gate sequence into both arms.
  const uint32_t flags = Sched::kFixedFlags >= 0
                             ? (A.flags & PF_INIT) | (uint32_t)Sched::kFixedFlags
                             : A.flags;
  uint32_t base, off[NA];
  // Psi_0 is read in logical order; the passes' own states in their layouts
  const bool logical_in = !BWD && !(flags & PF_INIT) && A.psi0_in;
  io_offsets<R>(logical_in ? A.io_lin : A.io, A.k, A.ng, tid, g, base, off);
  const size_t sbase = (size_t)b << (A.k + A.ng);
  const uint32_t sbytes = 8u << (A.k + A.ng);
  // the register columns of the layout this pass writes, read before the gate
  // sequence (its barriers would make a later read a per-lane one)
  uint32_t oc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) oc[r] = A.io_out[A.k - R + r];
  St<R> a, l;
  if (!BWD && (flags & PF_INIT)) {
    if constexpr (Sched::kProductStart) {
      Sched::template product_start<R>(a, w);  // the state after the heads
    } else {
#pragma unroll
      for (int j = 0; j < NA; ++j) {
        a.r[j] = 0.f;
        a.i[j] = 0.f;
      }
      if (tid == 0 && g == 0) a.r[0] = 1.f;
    }
  } else {
    load_tile<R>(a, state_rsrc(reinterpret_cast<const float2*>(A.psi_src) + sbase, sbytes), base,
                 off);
  }
  if (BWD) {
    if (flags & PF_MAKE_LAMBDA) {
      make_lambda<R, Sched>(l, a, A.grad_out + b * A.n, A.n, A.start_phys, A.zmask, w.tb, true,
                            Sched::esigns(w));
    } else {
      load_tile<R>(l, state_rsrc(reinterpret_cast<const float2*>(A.lam_src) + sbase, sbytes),
                   base, off);
    }
  }

  Sched::template run<R, BWD, true>(a, l, w, A.ins, A.n_ins);

  // the stores, in the layout this pass writes
  io_offsets<R>(A.io_out, A.k, A.ng, tid, g, base, off);
#pragma unroll
  for (int j = 0; j < NA; ++j) off[j] = xor_cols<R>(j, oc);
  const uint32_t base_b = opaque(base) << 3;
  // the adjoint stores lambda only (its psi is the state the forward saved at
  // this pass's start), and nothing at all in its last pass
  if (!BWD) {
    const auto dst = state_rsrc(reinterpret_cast<float2*>(A.psi_dst) + sbase, sbytes);
#pragma unroll
    for (int j = 0; j < NA; ++j) amp_store(dst, base_b, off[j], a.r[j], a.i[j]);
  }
  if (BWD) {
    if (!(flags & PF_LAST_ADJ)) {
      const auto dst = state_rsrc(reinterpret_cast<float2*>(A.lam_dst) + sbase, sbytes);
#pragma unroll
      for (int j = 0; j < NA; ++j) amp_store(dst, base_b, off[j], l.r[j], l.i[j]);
    }
    if constexpr (Sched::kHeadPartials) {
      // lambda where the heads end, contracted against the heads' states
      if (flags & PF_LAST_ADJ) Sched::template head_partials<WG, R>(l, w, A.vpart + blk * Sched::kNV);
    }
    __syncthreads();
    float* gp = A.gpart + blk * A.n_slots;
    for (int i = tid; i < A.n_pslots; i += WG) {
      float v = 0.f;
      for (int r = 0; r < G; ++r) v += acc[i * G + r];
      gp[A.pslots[i]] += v;
    }
  } else if (flags & PF_ZPART) {
    if (A.probs) {
      // the tile's rows are in logical order: a permutation of the stored
      // state's addresses, so the stores stay coalesced
      const uint32_t xm = frame_xmask(Sched::esigns(w), A.n);
      float* pd = A.probs + sbase;
      io_offsets<R>(A.io_lout, A.k, A.ng, tid, g, base, off);
#pragma unroll
      for (int j = 0; j < NA; ++j) pd[(base ^ off[j]) ^ xm] = a.r[j] * a.r[j] + a.i[j] * a.i[j];
    }
    float* ez = xbuf;
    z_partials<R, Sched>(a, ez, A.n, A.end_phys, A.zmask, w);
    for (int q = tid; q < A.n; q += WG) {
      float e = 0.f;
      for (int r = 0; r < G; ++r) e += ez[q * G + r];
      A.epart[blk * A.n + q] = e;
    }
  }
}

}  // namespace vqc
