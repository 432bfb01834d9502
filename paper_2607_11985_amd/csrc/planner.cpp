// planner.cpp -- compile phase (Algorithm 1, compile phase): validate the
// static gate list, lower it to primitives, classify every angle as parametric
// (param / input slot) or constant (cached cos/sin), and plan the register-tile
// schedule of the forward sweep and of the adjoint (reverse) sweep.
//
// Host-only code: no device calls, so it can run (and be tested) without a GPU.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>

#include "vqc.h"
#include "vqc_internal.h"

namespace vqc {
namespace {

struct Mapping {
  int k = 0;
  int p2q[kMaxTileQubits];
  int q2p[kMaxQubits];
};

// Qubit a primitive needs on a register bit, or -1 (diagonal gates and CNOT
// controls work from any physical bit).
int register_need(const Prim& p) {
  switch (p.kind) {
    case P_RX:
    case P_RY:
      return p.q0;
    case P_CNOT:
      return p.q1;
    default:
      return -1;
  }
}

// next_need[i * nq + q]: first index >= i of `seq` that needs q on a register.
std::vector<int> next_need_table(const std::vector<Prim>& seq, int nq) {
  const int G = (int)seq.size();
  std::vector<int> t((size_t)(G + 1) * nq, INT_MAX);
  for (int i = G - 1; i >= 0; --i) {
    for (int q = 0; q < nq; ++q) t[(size_t)i * nq + q] = t[(size_t)(i + 1) * nq + q];
    const int need = register_need(seq[i]);
    if (need >= 0) t[(size_t)i * nq + need] = i;
  }
  return t;
}

// Exchange tables.  The LDS slot of an amplitude is a GF(2)-linear function
// lam(x) of its logical tile index; lam is chosen per exchange so that the
// lanes of a 32-lane group hit 32 distinct 8-byte slots modulo 256 bytes both
// when writing in the old layout and when reading in the new one:
// slot bit i (i < bank bits) = x[old lane-i qubit] xor x[new lane-i qubit]
// (the second term only when the qubit changes), the other qubits get one
// high bit each.  Exchanges only swap register bits with thread bits, so a
// qubit never moves between two lane positions, which keeps lam bijective.
int emit_exchange(const Mapping& a, const Mapping& b, int k, int t, std::vector<uint32_t>& cols,
                  std::string& msg) {
  const int lb = std::min(kBankBits, t);
  uint32_t lam[kMaxQubits];
  bool in_a[kMaxQubits], in_b[kMaxQubits];
  std::memset(lam, 0, sizeof(lam));
  std::memset(in_a, 0, sizeof(in_a));
  std::memset(in_b, 0, sizeof(in_b));
  for (int i = 0; i < lb; ++i) {
    in_a[a.p2q[kRegBits + i]] = true;
    in_b[b.p2q[kRegBits + i]] = true;
  }
  for (int i = 0; i < lb; ++i) {
    const int qa = a.p2q[kRegBits + i], qb = b.p2q[kRegBits + i];
    lam[qa] |= 1u << i;
    if (qb != qa) {
      if (in_a[qb] || in_b[qa]) {
        msg = "internal: exchange moves a qubit between lane positions";
        return VQC_ERR_UNSUPPORTED;
      }
      lam[qb] |= 1u << i;
    }
  }
  int nb = lb;
  for (int p = 0; p < k; ++p) {
    const int q = a.p2q[p];
    if (!in_a[q]) lam[q] |= 1u << nb++;
  }
  if (nb != k) {
    msg = "internal: exchange layout is not a bijection";
    return VQC_ERR_UNSUPPORTED;
  }
  const int off = (int)cols.size();
  for (int p = 0; p < k; ++p) cols.push_back(lam[a.p2q[p]]);
  for (int p = 0; p < k; ++p) cols.push_back(lam[b.p2q[p]]);
  return off;
}

void emit(std::vector<uint32_t>& out, uint32_t op, int a, int b, uint32_t arg) {
  out.push_back(ins_word0(op, (uint32_t)a, (uint32_t)b));
  out.push_back(arg);
}

// One sweep over `seq` starting from mapping `m` (updated to the end mapping).
int plan_sweep(const std::vector<Prim>& seq, int nq, int k, int t, Mapping& m,
               std::vector<uint32_t>& out, std::vector<uint32_t>& cols, int& exchanges,
               std::string& msg) {
  const std::vector<int> nn = next_need_table(seq, nq);
  for (size_t i = 0; i < seq.size(); ++i) {
    const Prim& pr = seq[i];
    const int need = register_need(pr);
    if (need >= 0 && m.q2p[need] >= kRegBits) {
      // Belady: the register bits get the kRegBits qubits needed soonest.
      std::vector<int> qs;
      for (int q = 0; q < nq; ++q)
        if (m.q2p[q] >= 0) qs.push_back(q);
      const int* row = &nn[i * (size_t)nq];
      std::stable_sort(qs.begin(), qs.end(), [&](int x, int y) {
        if (row[x] != row[y]) return row[x] < row[y];
        const bool rx = m.q2p[x] < kRegBits, ry = m.q2p[y] < kRegBits;
        if (rx != ry) return rx;  // keep residents on ties
        return x < y;
      });
      bool chosen[kMaxQubits] = {false};
      for (int r = 0; r < kRegBits; ++r) chosen[qs[r]] = true;
      std::vector<int> incoming, outgoing;
      for (int r = 0; r < kRegBits; ++r)
        if (!chosen[m.p2q[r]]) outgoing.push_back(r);
      for (int r = 0; r < kRegBits; ++r)
        if (m.q2p[qs[r]] >= kRegBits) incoming.push_back(qs[r]);
      Mapping nm = m;
      for (size_t j = 0; j < incoming.size(); ++j) {
        const int qin = incoming[j];
        const int pin = m.q2p[qin];
        const int pout = outgoing[j];
        const int qout = m.p2q[pout];
        nm.p2q[pout] = qin;
        nm.q2p[qin] = pout;
        nm.p2q[pin] = qout;
        nm.q2p[qout] = pin;
      }
      const int off = emit_exchange(m, nm, k, t, cols, msg);
      if (off < 0) return off;
      emit(out, OP_EXCHANGE, 0, 0, (uint32_t)off);
      ++exchanges;
      m = nm;
    }
    switch (pr.kind) {
      case P_RX: emit(out, OP_RX, m.q2p[pr.q0], 0, (uint32_t)pr.occ); break;
      case P_RY: emit(out, OP_RY, m.q2p[pr.q0], 0, (uint32_t)pr.occ); break;
      case P_RZ: emit(out, OP_RZ, m.q2p[pr.q0], 0, (uint32_t)pr.occ); break;
      case P_CNOT: emit(out, OP_CNOT, m.q2p[pr.q0], m.q2p[pr.q1], 0); break;
      case P_CZ: emit(out, OP_CZ, m.q2p[pr.q0], m.q2p[pr.q1], 0); break;
      default: msg = "internal: unknown primitive"; return VQC_ERR_UNSUPPORTED;
    }
  }
  return 0;
}

int n_angles(int kind) {
  if (kind == VQC_RX || kind == VQC_RY || kind == VQC_RZ) return 1;
  if (kind == VQC_ROT) return 3;
  return 0;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

int build_plan(const std::vector<HostOp>& ops, int n, int P, int F, int path, Plan& plan,
               std::string& msg) {
  if (n < 1 || n > kMaxQubits) {
    msg = "n_qubits must be in [1, " + std::to_string(kMaxQubits) + "]";
    return n < 1 ? VQC_ERR_INVALID_ARG : VQC_ERR_TOO_LARGE;
  }
  if (P < 0 || F < 0) {
    msg = "n_params and n_inputs must be >= 0";
    return VQC_ERR_INVALID_ARG;
  }
  plan = Plan();
  plan.n = n;
  plan.P = P;
  plan.F = F;
  plan.n_ops = (int)ops.size();
  // validation and lowering (Sec. 3 "Static Circuit Scope": gate identity and
  // wiring are fixed here; only angles vary at run time)
  for (size_t k = 0; k < ops.size(); ++k) {
    const HostOp& o = ops[k];
    const std::string at = "op " + std::to_string(k) + ": ";
    if (o.kind < VQC_RX || o.kind > VQC_CZ) {
      msg = at + "unknown kind " + std::to_string(o.kind);
      return VQC_ERR_INVALID_ARG;
    }
    if (o.w0 < 0 || o.w0 >= n) {
      msg = at + "wire " + std::to_string(o.w0) + " out of range";
      return VQC_ERR_INVALID_ARG;
    }
    if (o.kind == VQC_CNOT || o.kind == VQC_CZ) {
      if (o.w1 < 0 || o.w1 >= n) {
        msg = at + "second wire " + std::to_string(o.w1) + " out of range";
        return VQC_ERR_INVALID_ARG;
      }
      if (o.w1 == o.w0) {
        msg = at + "two-qubit gate on a single wire";
        return VQC_ERR_INVALID_ARG;
      }
      plan.prims.push_back({o.kind == VQC_CNOT ? P_CNOT : P_CZ, o.w0, o.w1, -1});
      continue;
    }
    const int na = n_angles(o.kind);
    int occ0 = (int)plan.occ_src.size();
    for (int s = 0; s < na; ++s) {
      const int src = o.src[s], idx = o.idx[s];
      if (src == VQC_SRC_PARAM) {
        if (idx < 0 || idx >= P) {
          msg = at + "param index " + std::to_string(idx) + " out of range";
          return VQC_ERR_INVALID_ARG;
        }
      } else if (src == VQC_SRC_INPUT) {
        if (idx < 0 || idx >= F) {
          msg = at + "input index " + std::to_string(idx) + " out of range";
          return VQC_ERR_INVALID_ARG;
        }
      } else if (src != VQC_SRC_CONST) {
        msg = at + "unknown angle source " + std::to_string(src);
        return VQC_ERR_INVALID_ARG;
      } else if (!std::isfinite(o.val[s])) {
        msg = at + "constant angle is not finite";
        return VQC_ERR_INVALID_ARG;
      }
      plan.occ_src.push_back(src);
      plan.occ_idx.push_back(src == VQC_SRC_CONST ? 0 : idx);
      plan.occ_slot.push_back(src == VQC_SRC_PARAM ? idx : src == VQC_SRC_INPUT ? P + idx : -1);
      // constant gates are cached at compile time (Algorithm 1, compile phase)
      const double half = 0.5 * (double)o.val[s];
      plan.occ_cs.push_back(src == VQC_SRC_CONST ? (float)std::cos(half) : 0.f);
      plan.occ_cs.push_back(src == VQC_SRC_CONST ? (float)std::sin(half) : 0.f);
    }
    if (o.kind == VQC_ROT) {
      // ROT(phi, theta, omega) = RZ(omega) RY(theta) RZ(phi): phi first
      plan.prims.push_back({P_RZ, o.w0, -1, occ0 + 0});
      plan.prims.push_back({P_RY, o.w0, -1, occ0 + 1});
      plan.prims.push_back({P_RZ, o.w0, -1, occ0 + 2});
    } else {
      const int pk = o.kind == VQC_RX ? P_RX : o.kind == VQC_RY ? P_RY : P_RZ;
      plan.prims.push_back({pk, o.w0, -1, occ0});
    }
  }
  const int n_occ = (int)plan.occ_src.size();
  const int nq = std::max(n, kRegBits);  // qubits >= n stay |0> and are never read
  plan.nq = nq;
  if (path == VQC_PATH_AUTO) path = nq <= kMaxTileQubits ? VQC_PATH_RESIDENT : VQC_PATH_STREAM;
  if (path == VQC_PATH_STREAM) {
    msg = "the streaming path (n > 14) is not available in this build";
    return VQC_ERR_UNSUPPORTED;
  }
  if (path != VQC_PATH_RESIDENT) {
    msg = "unknown path option";
    return VQC_ERR_INVALID_ARG;
  }
  if (nq > kMaxTileQubits) {
    msg = "the resident path holds at most 14 qubits";
    return VQC_ERR_UNSUPPORTED;
  }
  plan.path = VQC_PATH_RESIDENT;
  plan.k = nq;
  plan.t = nq - kRegBits;
  const int T = 1 << plan.t;
  plan.WG = std::max(64, T);
  plan.S = plan.WG / T;
  plan.G = T >= 64 ? plan.WG / 64 : plan.S;

  // initial mapping: registers get the first qubits the sweep needs there
  Mapping m;
  m.k = plan.k;
  for (int q = 0; q < kMaxQubits; ++q) m.q2p[q] = -1;
  {
    const std::vector<int> nn = next_need_table(plan.prims, nq);
    std::vector<int> qs(nq);
    for (int q = 0; q < nq; ++q) qs[q] = q;
    std::stable_sort(qs.begin(), qs.end(), [&](int x, int y) { return nn[x] < nn[y]; });
    std::vector<int> rest(qs.begin() + kRegBits, qs.end());
    std::sort(rest.begin(), rest.end());
    for (int r = 0; r < kRegBits; ++r) {
      m.p2q[r] = qs[r];
      m.q2p[qs[r]] = r;
    }
    for (size_t j = 0; j < rest.size(); ++j) {
      m.p2q[kRegBits + j] = rest[j];
      m.q2p[rest[j]] = kRegBits + (int)j;
    }
  }
  int rc = plan_sweep(plan.prims, nq, plan.k, plan.t, m, plan.fwd, plan.cols, plan.fwd_exchanges,
                      msg);
  if (rc < 0) return rc;
  plan.end_phys.assign(nq, 0);
  for (int q = 0; q < nq; ++q) plan.end_phys[q] = (uint8_t)m.q2p[q];
  std::vector<Prim> rev(plan.prims.rbegin(), plan.prims.rend());
  rc = plan_sweep(rev, nq, plan.k, plan.t, m, plan.bwd, plan.cols, plan.bwd_exchanges, msg);
  if (rc < 0) return rc;

  // LDS: exchange buffer | angle table [occ][S] | gradient accumulators [slot][G]
  const size_t xbuf = (size_t)plan.WG * kRegAmps * 8;
  plan.lds_tab = xbuf;
  const size_t tab = align_up((size_t)n_occ * plan.S * 8, 16);
  plan.lds_acc = xbuf + tab;
  const size_t acc = align_up((size_t)(P + F) * plan.G * 4, 16);
  plan.lds_fwd = std::max<size_t>(xbuf + tab, 16);
  plan.lds_bwd = xbuf + tab + acc;
  if (plan.lds_bwd > (size_t)kLdsBytes) {
    msg = "circuit too large for on-chip tables: " + std::to_string(plan.lds_bwd) +
          " bytes of LDS needed (limit " + std::to_string(kLdsBytes) + ")";
    return VQC_ERR_TOO_LARGE;
  }
  return 0;
}

}  // namespace vqc
