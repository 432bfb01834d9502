// jit.cpp -- compile once: the circuit's schedule becomes straight-line gfx950
// code (Sec. 3 "Compile-Once Lowering and Execution").
//
// The planner's instruction streams are turned into source text in which every
// register position, exchange layout and gradient slot is a literal: a gate is a
// call of the register-tile template for its position, a CNOT between register
// bits is a renaming, and exchanges use constant column tables.  The text plus
// the shared device code (vqc_device.h) is compiled with hiprtc for gfx950, one
// program per kernel, several at a time in helper processes, and loaded as
// modules; launches go through hipModuleLaunchKernel.  Identical kernels are
// compiled once per process.
#include <dlfcn.h>
#include <fcntl.h>
#include <hip/hip_runtime_api.h>
#include <spawn.h>
#include <sys/wait.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <functional>
#include <map>
#include <memory>
#include <mutex>
#include <sstream>
#include <thread>

#include "vqc.h"
#include "vqc_internal.h"

extern char** environ;

namespace vqc {

namespace {

std::string hex(uint32_t v) {
  char b[16];
  std::snprintf(b, sizeof b, "0x%xu", v);
  return b;
}

std::string hex64(uint64_t v) {
  char b[24];
  std::snprintf(b, sizeof b, "0x%llxull", (unsigned long long)v);
  return b;
}

// How the adjoint kernels collect gradient partials.  Lanes are grouped by
// sample (tm lanes: the sample's threads, at most one wave).  With `regs`, lane
// j of a group keeps slots j, j + tm, ... in registers (nr of them) and adds
// the group sum of each rotation's partial to the owning lane: no branch and no
// LDS access per rotation.  Otherwise one lane adds it to the LDS accumulator.
struct GradMode {
  int tm = 64, ns = 0, nr = 0;
  bool regs = false;
};
constexpr int kMaxGradRegs = 16;

GradMode grad_mode(int lanes_per_sample, int n_slots) {
  GradMode g;
  g.tm = lanes_per_sample < 64 ? lanes_per_sample : 64;
  g.ns = n_slots;
  g.nr = (n_slots + g.tm - 1) / g.tm;
  g.regs = g.nr <= kMaxGradRegs;
  return g;
}

// ------------------------------------------------------------ tangent form
// With one sample per workgroup the generated kernels apply every rotation as
// I - i t P with |t| <= 1 (vqc_device.h, "tangent form"): the Pauli P^m that
// brings the half angle into [-pi/4, pi/4] is moved aside.  The moved Paulis
// form a frame F, one Pauli string per sample, which changes where a rotation's
// m is odd (its parity bit) and where an entangler conjugates it.  That is
// GF(2)-linear, so for rotation j, "F anticommutes with P_j on j's qubit" (then
// t_j and the gradient of j change sign) is the parity of (parities AND
// arow[j]), and "<Z_q> changes sign" that of (parities AND erow[q]); the rows
// are compile-time constants over all occurrences in circuit order.  Gates that
// the streaming planner reorders commute, and a Pauli carried through a
// commuting gate is unchanged, so the rows hold for every execution order.
// The factors cos(phi') are applied to the state after every kBlock rotations
// of a stream and at its end (each unscaled gate grows the state by at most
// sqrt 2, so a block grows it by at most 2^32, far inside the float range), and
// the adjoint scales each gradient by the square of the factors not yet
// applied (at least 2^-64).
constexpr int kBlock = 64;

struct Frame {
  int words = 0;
  std::vector<uint32_t> arow;  // [occ][words]
  std::vector<uint32_t> erow;  // [qubit][words]
};

void pauli_bits(int kind, uint32_t& x, uint32_t& z) {
  x = kind == P_RX || kind == P_RY;
  z = kind == P_RY || kind == P_RZ;
}

Frame frame_rows(const Plan& p) {
  // the circuit in an order equivalent to the original: the gates run, then the
  // trailing entanglers folded into the measurement (the rows describe the
  // frame on the final state)
  std::vector<Prim> all(p.prims);
  all.insert(all.end(), p.tail.begin(), p.tail.end());
  Frame f;
  const int nocc = (int)p.occ_src.size();
  f.words = (nocc + 31) / 32;
  const int W = f.words;
  f.arow.assign((size_t)nocc * W, 0u);
  f.erow.assign((size_t)p.n * W, 0u);
  for (size_t i = 0; i < all.size(); ++i) {
    const Prim& src = all[i];
    if (src.occ < 0) continue;
    const int k = src.occ;
    uint32_t px, pz;
    pauli_bits(src.kind, px, pz);
    uint32_t x = px << src.q0, z = pz << src.q0;
    for (size_t j = i + 1; j < all.size(); ++j) {
      const Prim& g = all[j];
      if (g.kind == P_CNOT) {  // X_c -> X_c X_t, Z_t -> Z_c Z_t
        const uint32_t xc = (x >> g.q0) & 1u, zt = (z >> g.q1) & 1u;
        x ^= xc << g.q1;
        z ^= zt << g.q0;
      } else if (g.kind == P_CZ) {  // X_a -> X_a Z_b
        const uint32_t xa = (x >> g.q0) & 1u, xb = (x >> g.q1) & 1u;
        z ^= (xa << g.q1) | (xb << g.q0);
      } else {
        uint32_t gx, gz;
        pauli_bits(g.kind, gx, gz);
        const uint32_t anti = (((x >> g.q0) & 1u) & gz) ^ (((z >> g.q0) & 1u) & gx);
        if (anti) f.arow[(size_t)g.occ * W + (k >> 5)] |= 1u << (k & 31);
      }
    }
    for (int q = 0; q < p.n; ++q)
      if ((x >> q) & 1u) f.erow[(size_t)q * W + (k >> 5)] |= 1u << (k & 31);
  }
  return f;
}

std::vector<int> stream_rotations(const uint32_t* ins, int n_ins) {
  std::vector<int> occ;
  for (int pc = 0; pc < n_ins; ++pc) {
    const int op = ins[2 * pc] & 31;
    if (op == OP_RX || op == OP_RY || op == OP_RZ) occ.push_back((int)ins[2 * pc + 1]);
  }
  return occ;
}


// Tables of one kernel, in LDS after the kernel's own layout.
struct TanMode {
  bool on = false;
  int W = 0;
  std::vector<int> focc, bocc;  // rotations of the forward / adjoint stream, in stream order
  bool esign = false;
  size_t off_bits = 0, off_gm = 0, off_es = 0, end = 0;
};

size_t align16(size_t v) { return (v + 15) / 16 * 16; }

TanMode tan_mode(const Plan& p, const uint32_t* fins, int fn, const uint32_t* bins, int bn, int S,
                 bool esign, size_t base) {
  TanMode t;
  const int nocc = (int)p.occ_src.size();
  t.W = std::max(1, (nocc + 31) / 32);
  if (fins) t.focc = stream_rotations(fins, fn);
  if (bins) t.bocc = stream_rotations(bins, bn);
  t.esign = esign;
  size_t off = align16(base);
  t.off_bits = off;
  off = align16(off + (size_t)(t.W + 1) * 4);  // + 1: the ballot writes word pairs
  t.off_gm = off;
  if (bins) off = align16(off + (size_t)nocc * 4);
  t.off_es = off;
  if (esign) off = align16(off + (size_t)p.n * 4);
  t.end = off;
  t.on = S == 1 && t.end <= (size_t)kLdsBytes;
  return t;
}

template <typename T>
void emit_array(std::ostringstream& o, const char* type, const char* name, const std::vector<T>& v) {
  o << "  static constexpr " << type << " " << name << "[] = {";
  if (v.empty()) o << "0";
  for (size_t i = 0; i < v.size(); ++i) o << (i ? "," : "") << (uint64_t)v[i];
  o << "};\n";
}

// prepare(): (cos, sin)(theta/2) -> (t, cos phi') in place with the parity bits
// (one ballot per 64 occurrences), then in one round over the streams'
// rotations: the frame sign of each (t negated in place, once) and the sign
// of the adjoint's gradients; and the <Z> signs.  esigns(): those signs.  The
// block factors are products the schedule forms as it goes (bp).
void emit_tables(std::ostringstream& o, const Plan& p, const TanMode& t, const Frame& fr,
                 int nt, bool all = false, bool load = false,
                 const std::vector<char>* head = nullptr) {
  const int nocc = (int)p.occ_src.size(), W = t.W;
  o << "static constexpr bool kLoadTables = " << (t.on && load ? "true" : "false") << ";\n"
    << "static constexpr uint32_t kOffGm = " << t.off_gm << "u;\n";
  if (!t.on) {
    o << "struct Pre {};\n"
      << "__device__ __forceinline__ static Pre preload(int) { return Pre(); }\n"
      << "__device__ __forceinline__ static void prepare(const Walk&, int, int, const Pre&) {}\n"
      << "__device__ __forceinline__ static const float* esigns(const Walk&) { return nullptr; }\n";
    return;
  }
  if (load) {
    // the pass reads the sample's tables that the table kernel wrote
    o << "__device__ __forceinline__ static void load_tables(const Walk& w, const PassArgs& A, "
         "int64_t b, int tid, int nt) {\n"
      << "  float2* tab = const_cast<float2*>(w.tab);\n"
      << "  const float2* T = reinterpret_cast<const float2*>(A.tabs) + b * " << nocc << ";\n"
      << "  for (int i = tid; i < " << nocc << "; i += nt) tab[i] = T[i];\n";
    if (!t.bocc.empty())
      o << "  float* gm = reinterpret_cast<float*>(w.smem + " << t.off_gm << "u);\n"
        << "  const float* G = A.gsig + b * " << nocc << ";\n"
        << "  for (int i = tid; i < " << nocc << "; i += nt) gm[i] = G[i];\n";
    if (t.esign)
      o << "  float* es = reinterpret_cast<float*>(w.smem + " << t.off_es << "u);\n"
        << "  for (int q = tid; q < " << p.n << "; q += nt) es[q] = A.esig[b * " << p.n
        << " + q];\n";
    o << "}\n";
  }
  // instances: the forward stream's rotations, then the adjoint's
  std::vector<int> inst = t.focc;
  inst.insert(inst.end(), t.bocc.begin(), t.bocc.end());
  std::vector<uint32_t> rows;
  for (int k : inst)
    for (int j = 0; j < W; ++j)
      rows.push_back(j < fr.words ? fr.arow[(size_t)k * fr.words + j] : 0u);
  std::vector<uint32_t> erows;
  if (t.esign)
    for (int q = 0; q < p.n; ++q)
      for (int j = 0; j < W; ++j)
        erows.push_back(j < fr.words ? fr.erow[(size_t)q * fr.words + j] : 0u);
  const int nf = (int)t.focc.size(), ni = (int)inst.size();
  // preload(): each thread's entries of the constant rows, read before the
  // angle table (their latency then overlaps its loads) when they fit in a
  // few registers; prepare() reads them in place otherwise
  const int ri = (ni + nt - 1) / nt, re = t.esign ? (p.n + nt - 1) / nt : 0;
  const int nreg = ri * (1 + W) + re * W;
  const bool pre = ni > 0 && nreg <= 48;
  o << "struct Pre {";
  if (pre) o << " uint32_t o[" << ri << "], r[" << ri * W << "], e[" << std::max(re * W, 1) << "];";
  o << " };\n"
    << "__device__ __forceinline__ static Pre preload(int tid) {\n"
    << "  Pre p;\n";
  if (pre) {
    emit_array(o, "uint16_t", "kOcc", inst);
    emit_array(o, "uint32_t", "kArow", rows);
    o << "#pragma unroll\n"
      << "  for (int r = 0; r < " << ri << "; ++r) {\n"
      << "    const int i = min(r * " << nt << " + tid, " << ni - 1 << ");\n"
      << "    p.o[r] = kOcc[i];\n"
      << "#pragma unroll\n"
      << "    for (int j = 0; j < " << W << "; ++j) p.r[r * " << W << " + j] = kArow[i * " << W
      << " + j];\n"
      << "  }\n";
    if (re > 0) {
      emit_array(o, "uint32_t", "kErow", erows);
      o << "#pragma unroll\n"
        << "  for (int r = 0; r < " << re << "; ++r) {\n"
        << "    const int q = min(r * " << nt << " + tid, " << p.n - 1 << ");\n"
        << "#pragma unroll\n"
        << "    for (int j = 0; j < " << W << "; ++j) p.e[r * " << W << " + j] = kErow[q * " << W
        << " + j];\n"
        << "  }\n";
    }
  } else {
    o << "  (void)tid;\n";
  }
  o << "  return p;\n}\n";
  if (head) {
    // whether occurrence i0 + tid is a head rotation: one 64-bit mask per 64
    // occurrences, picked by the wave-uniform chunk index
    o << "__device__ __forceinline__ static bool head_occ(int i0, int tid) {\n"
      << "  const uint32_t c = (uint32_t)(i0 >> 6) + "
         "__builtin_amdgcn_readfirstlane((uint32_t)tid >> 6);\n"
      << "  uint64_t m = 0ull;\n";
    for (int c = 0; 64 * c < nocc; ++c) {
      uint64_t m = 0;
      for (int j = 0; j < 64 && 64 * c + j < nocc; ++j)
        if ((*head)[64 * c + j]) m |= 1ull << j;
      if (m) o << "  if (c == " << c << "u) m = " << hex64(m) << ";\n";
    }
    o << "  return (m >> (tid & 63)) & 1ull;\n}\n";
  }
  o << "__device__ __forceinline__ static void prepare(const Walk& w, int tid, int nt, "
       "const Pre& pre) {\n"
    << "  (void)pre;\n"
    << "  float2* tab = const_cast<float2*>(w.tab);\n"
    << "  float* tx = reinterpret_cast<float*>(tab);  // tab[k].x = tx[2 k]\n"
    << "  uint32_t* bits = reinterpret_cast<uint32_t*>(w.smem + " << t.off_bits << "u);\n"
    << "  for (int i0 = 0; i0 < " << nocc << "; i0 += nt) {\n"
    << "    const int i = i0 + tid;\n"
    << "    bool odd = false;\n"
    // head rotations run exactly (their parity stays 0, their (cos, sin) stay)
    << "    if (i < " << nocc << (head ? " && !head_occ(i0, tid)" : "") << ") {\n"
    << "      const float2 cs = tab[i];\n"
    << "      odd = fabsf(cs.y) > fabsf(cs.x);\n"
    << "      tab[i] = make_float2(odd ? -cs.x / cs.y : cs.y / cs.x, odd ? fabsf(cs.y) : fabsf(cs.x));\n"
    << "    }\n"
    << "    const uint64_t m = __ballot(odd);\n"
    << "    if ((tid & 63) == 0 && i < " << nocc << ") {\n"
    << "      bits[i >> 5] = (uint32_t)m;\n"
    << "      bits[(i >> 5) + 1] = (uint32_t)(m >> 32);\n"
    << "    }\n"
    << "  }\n"
    << "  __syncthreads();\n";
  if (!pre) {
    emit_array(o, "uint16_t", "kOcc", inst);
    emit_array(o, "uint32_t", "kArow", rows);
  }
  o << "  float* gm = reinterpret_cast<float*>(w.smem + " << t.off_gm << "u);\n"
    << "  (void)gm;\n"
    // a constant trip count, so that the rounds' table loads issue together
    << "#pragma unroll\n"
    << "  for (int i0 = 0; i0 < " << ni << "; i0 += nt) {\n"
    << "    const int i = i0 + tid;\n"
    << "    if (i < " << ni << ") {\n"
    << "    const bool f = i < " << nf << ";\n";
  if (pre)
    o << "    const int rr = i0 / " << nt << ";\n"
      << "    const int k = pre.o[rr];\n";
  else
    o << "    const int k = kOcc[i];\n";
  o << "    uint32_t par = 0u;\n"
    << "#pragma unroll\n"
    << "    for (int j = 0; j < " << W << "; ++j) par ^= __builtin_popcount(bits[j] & "
    << (pre ? "pre.r[rr * " + std::to_string(W) + " + j]"
            : "kArow[i * " + std::to_string(W) + " + j]")
    << ");\n"
    << "    if (f) {\n"
    << "      if (par & 1u) tx[2 * k] = -tx[2 * k];\n";
  if (all)  // the table kernel: every occurrence's t and gradient sign
    o << "      gm[k] = (par & 1u) ? -1.f : 1.f;\n";
  o << "    } else {\n";
  if (nf == 0)  // a lone adjoint stream applies the signs itself
    o << "      if (par & 1u) tx[2 * k] = -tx[2 * k];\n";
  o << "      gm[k] = (par & 1u) ? -1.f : 1.f;\n"
    << "    }\n"
    << "    }\n"
    << "  }\n";
  if (t.esign) {
    if (!pre) emit_array(o, "uint32_t", "kErow", erows);
    o << "#pragma unroll\n"
      << "  for (int q0 = 0; q0 < " << p.n << "; q0 += nt) {\n"
      << "    const int q = q0 + tid;\n"
      << "    if (q >= " << p.n << ") break;\n"
      << "    uint32_t par = 0u;\n"
      << "#pragma unroll\n"
      << "    for (int j = 0; j < " << W << "; ++j) par ^= __builtin_popcount(bits[j] & "
      << (pre ? "pre.e[(q0 / " + std::to_string(nt) + ") * " + std::to_string(W) + " + j]"
              : "kErow[q * " + std::to_string(W) + " + j]")
      << ");\n"
      << "    reinterpret_cast<float*>(w.smem + " << t.off_es << "u)[q] = (par & 1u) ? -1.f : 1.f;\n"
      << "  }\n";
  }
  o << "  __syncthreads();\n}\n";
  if (t.esign)
    o << "__device__ __forceinline__ static const float* esigns(const Walk& w) {\n"
      << "  return reinterpret_cast<const float*>(w.smem + " << t.off_es << "u);\n}\n";
  else
    o << "__device__ __forceinline__ static const float* esigns(const Walk&) { return nullptr; }\n";
}

// Batched gradient reduction for samples spanning whole waves.  A rotation's
// per-lane partial waits in pending register pd[slot % 16]; a batch is flushed
// when a position is needed by another slot, and at the end of the stream.
// The flush is a reduce-scatter over the 64 lanes: four halving steps pair
// lane bit b with value-index bit b (lane bit 2 through row_half_mirror, a
// lane ^ 7 pairing taken first while every lane still holds all values; then
// quad_perm 1032 and 2301 for bits 0 and 1, row_ror 8 for bit 3), leaving in
// each lane the partial of value lane % 16 over its 16-lane row; two more
// additions (a swizzle across 16 lanes, a shuffle across 32) complete it.
// The lane that owns the slot (lane = slot % 64) adds it to its register.
// About 4 instructions per rotation instead of a full DPP sum per rotation.
struct Pending {
  int tag[16];
  Pending() { clear(); }
  void clear() {
    for (int& t : tag) t = -1;
  }
  bool empty() const {
    for (int t : tag)
      if (t >= 0) return false;
    return true;
  }
};

// Whether an adjoint stream batches its gradient partials (emit_flush): the
// accumulator registers then hold slot 64 r + flush_slot(lane) in register r.
bool batched_flush(const Plan& p, bool bwd, const GradMode& gm, int R, int k) {
  return bwd && gm.regs && gm.tm == 64 && R <= 4 &&
         !(p.path == VQC_PATH_RESIDENT && (1 << (k - R)) > 512);
}

// Reduce-scatter of the 16 pending partials over the wave's 64 lanes.
// Position bit 3 pairs across lane bit 5 and bit 2 across lane bit 4, each
// pair one permlane swap (the upper half's first operand trades with the lower
// half's second) and one addition; bits 1 and 0 across lane bits 1 and 0, a
// select pair and a DPP addition each; then a sum over lane bits 2 and 3 (two
// DPP row rotations).  Lane L ends with the total of position
// (L5 L4 L1 L0) and adds it to slot 64 r + s when s % 16 is that position and
// s / 16 is (L3 L2): slot s of register r lives in lane
// (s3 s2 s5 s4 s1 s0), the layout the accumulators are written out in.
void emit_flush(std::ostringstream& o, Pending& pd) {
  if (pd.empty()) return;
  o << "  { float v[16];\n";
  for (int j = 0; j < 16; ++j)
    o << "    v[" << j << "] = " << (pd.tag[j] >= 0 ? "pd" + std::to_string(j) : "0.f") << ";\n";
  o << "    const uint32_t lo = opaque(ln);\n";
  // positions that may hold a partial, over the steps
  uint32_t used = 0;
  for (int j = 0; j < 16; ++j)
    if (pd.tag[j] >= 0) used |= 1u << j;
  auto swap_step = [&](int half, const char* fn) {
    uint32_t next = 0;
    for (int q = 0; q < half; ++q) {
      const bool a = (used >> q) & 1u, b = (used >> (q + half)) & 1u;
      if (!a && !b) continue;
      o << "    " << fn << "(v[" << q << "], v[" << q + half << "]); v[" << q << "] += v["
        << q + half << "];\n";
      next |= 1u << q;
    }
    used = next;
  };
  swap_step(8, "swap_pair32");  // position bit 3 <-> lane bit 5
  swap_step(4, "swap_pair16");  // position bit 2 <-> lane bit 4
  // position bit 1 <-> lane bit 1, then bit 0 <-> lane bit 0 (quad_perm 2301, 1032)
  static const int kDpp[2][3] = {{2, 1, 0x4E}, {1, 0, 0xB1}};
  for (const auto& st : kDpp) {
    const int half = st[0], lb = st[1], ctrl = st[2];
    uint32_t next = 0;
    o << "    { const bool hb = (lo >> " << lb << ") & 1u;\n";
    for (int q = 0; q < half; ++q) {
      const bool a = (used >> q) & 1u, b = (used >> (q + half)) & 1u;
      if (!a && !b) continue;
      o << "      const float k" << q << " = hb ? v[" << q + half << "] : v[" << q << "];\n"
        << "      const float s" << q << " = hb ? v[" << q << "] : v[" << q + half << "];\n"
        << "      v[" << q << "] = k" << q << " + dpp_f<" << ctrl << ">(s" << q << ");\n";
      next |= 1u << q;
    }
    o << "    }\n";
    used = next;
  }
  // lane bits 2 and 3: row_ror 4, row_ror 8
  o << "    float tot = v[0] + dpp_f<0x124>(v[0]);\n"
    << "    tot += dpp_f<0x128>(tot);\n";
  std::map<int, std::pair<uint32_t, uint32_t>> byreg;  // register -> (position mask, row table)
  for (int j = 0; j < 16; ++j) {
    if (pd.tag[j] < 0) continue;
    const int slot = pd.tag[j];
    auto& e = byreg[slot / 64];
    e.first |= 1u << j;
    e.second |= (uint32_t)((slot % 64) >> 4) << (2 * j);
  }
  o << "    const uint32_t j = (lo & 3u) | ((lo >> 2) & 12u), row = (lo >> 2) & 3u;\n";
  for (const auto& kv : byreg)
    o << "    ga[" << kv.first << "] += ((" << hex(kv.second.first) << " >> j) & 1u) && row == (("
      << hex(kv.second.second) << " >> (2u * j)) & 3u) ? tot : 0.f;\n";
  o << "  }\n";
  pd.clear();
}

// Whether exchange `arg` only swaps register bits with lane bits of the sample
// (bits the 64 lanes of one wave hold), and the (register bit, lane bit) pairs.
// The planner stores, after the exchange's 2k columns, where each physical
// bit's qubit goes.
bool lane_exchange(const Plan& p, uint32_t arg, int k, int R, int t,
                   std::vector<std::pair<int, int>>& swaps) {
  const int lanes = std::min(t, 6);
  const uint32_t* dest = p.cols.data() + arg + 2 * k;
  for (int q = 0; q < k; ++q) {
    const int d = (int)dest[q];
    if (d == q) continue;
    if (d < 0 || d >= k || (int)dest[d] != q) return false;  // not a transposition
    const int lo = std::min(q, d), hi = std::max(q, d);
    if (lo >= R || hi < R || hi - R >= lanes) return false;
    if (q == lo) swaps.push_back({lo, hi - R});
  }
  if (swaps.empty()) return false;
  // Lane bits 4 and 5 cost one permlane swap per two values.  Below that a
  // swap costs a DPP move (two for lane bit 2) and a select per value, more
  // VALU work than an LDS exchange of 8 or 16 amplitudes per thread: it pays
  // only where latency, not issue, bounds the kernel (4 amplitudes per thread;
  // measured: 35 % faster on the 8-qubit training step, 10 % slower on the
  // 12-qubit one).
  if (R <= 2) return true;
  for (const auto& sw : swaps)
    if (sw.second < 4) return false;
  return true;
}

// The chain-rule factor of an occurrence whose angle is mul * value + add, as
// a statement on the gradient partial g (nothing when mul is 1).
std::string occ_scale(const Plan& p, uint32_t occ) {
  if (!p.affine || p.occ_ma[2 * occ] == 1.f) return "";
  std::ostringstream o;
  o << " g *= " << std::hexfloat << (double)p.occ_ma[2 * occ] << "f;";
  return o.str();
}

// What a stream does with its swap frame at its end (vqc_device.h, "swap
// frame"): resolve it (the epilogue or the stores read positions; a pass's
// closing exchange has usually folded it already), or drop it (nothing reads
// the state).
enum FrameEnd { kFrameResolve, kFrameDrop };

// Statements of one instruction stream for register width R.  With tangent
// tables (tm.on) rotations use the tangent form and blocks are rescaled, and
// CNOTs from a thread / tile bit onto a register bit go to the swap frame.
// Whether a rotation joins a run of RZs applied as one diagonal: an RZ whose
// angle is not a constant.  A constant's float (cos, sin) pair is chosen so
// that the norm errors of the circuit's constant gates cancel one by one;
// in a product their rounding is the same every time the same gates come
// round and would add up instead.
bool fusable_rz(const Plan& p, uint32_t w0, uint32_t occ) {
  return (w0 & 31) == OP_RZ && p.occ_src[occ] != kSrcConst;
}

// Orders each stretch of single-qubit rotations (no entangler or exchange
// between them, so rotations on different bits commute) so that the fusable
// RZs on different bits come together: every such RZ at the head of its
// bit's sequence, then one other rotation from each bit, and again.  A Rot
// layer (RZ RY RZ on every qubit) becomes a run of RZs, the RYs, and another
// run of RZs.
std::vector<uint32_t> cluster_diagonals(const Plan& p, const uint32_t* ins, int n_ins) {
  std::vector<uint32_t> out(ins, ins + 2 * n_ins);
  auto is_rot = [&](int i) {
    const int op = ins[2 * i] & 31;
    return op == OP_RX || op == OP_RY || op == OP_RZ;
  };
  auto is_rz = [&](int i) { return fusable_rz(p, ins[2 * i], ins[2 * i + 1]); };
  for (int pc = 0; pc < n_ins;) {
    if (!is_rot(pc)) {
      ++pc;
      continue;
    }
    int end = pc;
    while (end < n_ins && is_rot(end)) ++end;
    std::map<int, std::vector<int>> seq;  // physical bit -> its rotations, in order
    for (int i = pc; i < end; ++i) seq[(ins[2 * i] >> 5) & 31].push_back(i);
    std::map<int, size_t> head;
    int w = pc;
    auto put = [&](int i) {
      out[2 * w] = ins[2 * i];
      out[2 * w + 1] = ins[2 * i + 1];
      ++w;
    };
    while (w < end) {
      for (auto& kv : seq) {
        size_t& h = head[kv.first];
        while (h < kv.second.size() && is_rz(kv.second[h])) put(kv.second[h++]);
      }
      for (auto& kv : seq) {
        size_t& h = head[kv.first];
        if (h < kv.second.size() && !is_rz(kv.second[h])) put(kv.second[h++]);
      }
    }
    pc = end;
  }
  return out;
}

void emit_schedule(std::ostringstream& o, const Plan& p, const uint32_t* ins, int n_ins, bool bwd,
                   int R, int k, int S, const GradMode& gm, const TanMode& tm,
                   const std::vector<char>* skip = nullptr, FrameEnd fend = kFrameResolve) {
  const int t = k - R;
  const bool tan = tm.on;
  // the swap frame: fs<r> (0 or 1 << 31 per thread) for register bit r; dirty:
  // the bits whose frame may be set here (known while generating)
  // (not in the kernels with gates on lane bits: there the lane swaps, which
  // would have to resolve the frame first, follow most CNOTs)
  const bool frames = tan && p.lanes == 0;
  // runs of RZs on different bits become one diagonal (emit_rz_run below;
  // one sample per workgroup, tangent form)
  const bool fuse = tan && S == 1 && R >= 2;
  std::vector<uint32_t> clustered;
  if (fuse) {
    clustered = cluster_diagonals(p, ins, n_ins);
    ins = clustered.data();
  }
  uint32_t dirty = 0;
  if (frames) {
    o << "  uint32_t";
    for (int r = 0; r < R; ++r) o << (r ? ", " : " ") << "fs" << r << " = 0u";
    o << ";\n";
  }
  // conditional swaps along the frame's bits in `bits` (one per state)
  auto resolve = [&](uint32_t bits) {
    bits &= dirty;
    for (int r = 0; r < R; ++r) {
      if (!((bits >> r) & 1u)) continue;
      o << "  cnot_tr<R, " << r << ">(a, fs" << r << " != 0u);";
      if (bwd) o << " cnot_tr<R, " << r << ">(l, fs" << r << " != 0u);";
      o << " fs" << r << " = 0u;\n";
    }
    dirty &= ~bits;
  };
  const int nrot = (int)(bwd ? tm.bocc.size() : tm.focc.size());
  int m = 0;  // rotation index in the stream
  // batched pending partials (a reduce-scatter per 16 slots instead of a DPP
  // sum per rotation).  With 16 amplitudes per thread the pending registers
  // sit beside psi and lambda: the streaming passes stay at 109-120 VGPRs, four
  // waves per SIMD (16-qubit adjoint 15 % fewer instructions, 1.93 -> 1.79
  // ms); the resident kernels go from four waves per SIMD to three (the
  // 12-qubit backward 110 -> 150 VGPRs) or stay at three (the 12-qubit step,
  // 168 VGPRs and the same spills) and still gain: step 0.879 -> 0.838 ms,
  // backward 0.666 -> 0.654 ms.  Not in 1024-thread workgroups (a 14-qubit
  // resident sample): those hold at most 128 VGPRs, and the pending registers
  // spilled 1.1 KiB per thread there (569 k -> 444 k evals/s).
  const bool batched = batched_flush(p, bwd, gm, R, k);
  Pending pend;
  if (batched)
    o << "  float pd0 = 0.f, pd1 = 0.f, pd2 = 0.f, pd3 = 0.f, pd4 = 0.f, pd5 = 0.f, pd6 = 0.f, "
         "pd7 = 0.f, pd8 = 0.f, pd9 = 0.f, pd10 = 0.f, pd11 = 0.f, pd12 = 0.f, pd13 = 0.f, "
         "pd14 = 0.f, pd15 = 0.f;\n";
  if (tan && bwd)
    o << "  const float* gmul = reinterpret_cast<const float*>(w.smem + " << tm.off_gm << "u);\n";
  if (tan)  // product of the factors cos(phi') of the current block so far
    o << "  float bp = 1.f;\n";
  // one sample per workgroup and 4 amplitudes per thread (latency-bound): the
  // angle table, and the adjoint's gradient signs, in registers (table_row)
  const bool sreg = S == 1 && R <= 2;
  // several samples per wave (small states): each lane reads its sample's
  // (cos, sin) of every rotation of the stream into registers at once, when
  // they are few, instead of one LDS read (and its latency) per gate
  std::vector<int> used;
  for (int pc = 0; pc < n_ins; ++pc) {
    const int op = ins[2 * pc] & 31;
    if (op == OP_RX || op == OP_RY || op == OP_RZ) used.push_back((int)ins[2 * pc + 1]);
  }
  std::sort(used.begin(), used.end());
  used.erase(std::unique(used.begin(), used.end()), used.end());
  const bool vreg = !tan && S > 1 && used.size() <= 32;
  if (vreg)
    for (int k : used)
      o << "  const float2 V" << k << " = w.tab[" << k << " * " << S << " + w.sl];\n";
  if (sreg) {
    int last = -1;
    for (int pc = 0; pc < n_ins; ++pc) {
      const int op = ins[2 * pc] & 31;
      if (op == OP_RX || op == OP_RY || op == OP_RZ) last = std::max(last, (int)ins[2 * pc + 1]);
    }
    for (int m = 0; 64 * m <= last; ++m) {
      o << "  const float2 T" << m << " = table_row(w, " << m << ", " << last << ");\n";
      if (tan && bwd)
        o << "  const float G" << m << " = table_row(gmul, " << m << ", " << last << ");\n";
    }
  }
  // The table entries of the next rotation are read one gate ahead (tangent
  // form, tables in LDS): each gate is its own basic block (gate_boundary),
  // so a read placed in the gate that uses it would leave the LDS latency
  // exposed at every rotation.
  std::vector<int> rots;
  for (int pc = 0; pc < n_ins; ++pc) {
    const int op = ins[2 * pc] & 31;
    const int occ = (int)ins[2 * pc + 1];
    if ((op == OP_RX || op == OP_RY || op == OP_RZ) && !(skip && (*skip)[occ])) rots.push_back(occ);
  }
  const bool ahead = tan && !sreg && !rots.empty();
  size_t ri = 0;  // the next rotation's index in rots
  if (ahead) {
    o << "  float2 tcn = w.tab[" << rots[0] << "];\n";
    if (bwd) o << "  float gmn = gmul[" << rots[0] << "];\n";
  }
  // The sample's thread bits, computed once in the 4-amplitude kernels: their
  // few waves leave registers to spare, and each lane-bit gate then skips
  // recomputing its bit (and the sign mask formed from it) from an opaque
  // copy of tb, which keeps the big kernels from holding masks across the
  // schedule.
  const bool hbits = R <= 2;
  if (hbits)
    for (int j = 0; j < t; ++j)
      o << "  const uint32_t hb" << j << " = (w.tb >> " << j << ") & 1u;\n";
  // a thread bit of the amplitude position (physical bit p >= R)
  auto bit = [&](int p) {
    return hbits ? "hb" + std::to_string(p - R) : "tile_bit<R>(w, " + std::to_string(p) + ")";
  };
  // A run of RZs (tangent form: amplitude x times 1 - i t z(x) per gate) is
  // one diagonal D: the forward multiplies each amplitude by D once.  The
  // adjoint takes every gradient of the run from Im(conj(lambda) psi), which
  // no diagonal gate changes (the tangent form scales it by 1 / cos^2 per
  // gate, which the block factor bp carries), then multiplies psi and lambda
  // by the inverse diagonal once.  D's entries (one per value of the run's
  // register bits, times the thread-bit factor) are formed in double,
  // depth first over those bits so that one product per level is live, and
  // each goes to float once.  A run is fused when an instruction count of
  // both ways says so, with a tenth of margin for the fused code's
  // registers.
  struct RzItem {
    int occ, bit, slot;
  };
  auto fused_cheaper = [&](const std::vector<RzItem>& run) {
    if (run.size() < 2) return false;
    const int N = 1 << R;
    int nt = 0, extra = 0;
    uint32_t B = 0;
    for (const auto& it : run) {
      if (it.bit >= R) ++nt;
      else {
        if ((B >> it.bit) & 1u) ++extra;
        B |= 1u << it.bit;
      }
    }
    const int mb = __builtin_popcount(B);
    int build = 2 * nt + 4 * extra;
    for (int i = 1; i < mb; ++i) build += 4 << (i - 1);
    if (mb) build += 4 << (mb - 1);
    const int states = bwd ? 2 : 1;
    const int fused = build + states * 4 * N + (bwd ? 3 * N + 3 * (int)run.size() : 0);
    const int sep = (int)run.size() * (bwd ? 6 : 2) * N;
    return 10 * fused < 9 * sep;
  };
  auto emit_rz_run = [&](const std::vector<RzItem>& run) {
    const int N = 1 << R, L = (int)run.size();
    const char* sg = bwd ? "" : "-";  // factor 1 + i sg x for z = +1
    o << "  { // " << L << " RZs as one diagonal\n";
    if (S == 1 && R <= 2) {  // the tables in registers (table_row)
      for (int i = 0; i < L; ++i) {
        const int occ = run[i].occ;
        o << "    const float2 tc" << i << " = table_entry<" << occ % 64 << ">(T" << occ / 64 << ");";
        if (bwd) o << " const float gm" << i << " = table_entry<" << occ % 64 << ">(G" << occ / 64 << ");";
        o << "\n";
      }
    } else {  // in LDS, the run's first entries read ahead
      if (rots[ri] != run[0].occ) o << "#error rotation prefetch out of order\n";
      for (int i = 0; i < L; ++i) {
        if (i == 0) {
          o << "    const float2 tc0 = tcn;";
          if (bwd) o << " const float gm0 = gmn;";
        } else {
          o << "    const float2 tc" << i << " = w.tab[" << run[i].occ << "];";
          if (bwd) o << " const float gm" << i << " = gmul[" << run[i].occ << "];";
        }
        o << "\n";
      }
      ri += L;
      if (ri < rots.size()) {
        o << "    tcn = w.tab[" << rots[ri] << "];";
        if (bwd) o << " gmn = gmul[" << rots[ri] << "];";
        o << "\n";
      }
    }
    uint32_t B = 0;
    int nt = 0;
    for (int i = 0; i < L; ++i) {
      const int b = run[i].bit;
      const bool neg = b < R && ((dirty >> b) & 1u);
      o << "    const float t" << i << " = "
        << (neg ? "flip_sign(tc" + std::to_string(i) + ".x, fs" + std::to_string(b) + ")"
                : "tc" + std::to_string(i) + ".x")
        << ";\n";
      if (b >= R) {
        // t times the thread's z on its bit
        o << "    const float z" << i << " = flip_sign(t" << i << ", " << bit(b) << " << 31);\n";
        ++nt;
      } else {
        B |= 1u << b;
      }
    }
    if (bwd) {
      // the gradients, all from Im(conj(lambda) psi) at the run's output
      for (int u = 0; u < N; ++u)
        o << "    const float I" << u << " = fmaf(-l.i[" << u << "], a.r[" << u << "], l.r[" << u
          << "] * a.i[" << u << "]);\n";
      std::vector<std::string> P(N);
      for (int u = 0; u < N; ++u) P[u] = "I" + std::to_string(u);
      for (int j = 0; j < R; ++j) {
        const int half = (int)P.size() / 2;
        if ((B >> j) & 1u) {  // sum over z on register bit j
          o << "    const float gb" << j << " = ";
          for (int w2 = 0; w2 < half; ++w2)
            o << (w2 ? " + " : "") << "(" << P[2 * w2] << " - " << P[2 * w2 + 1] << ")";
          o << ";\n";
        }
        if (!nt && !(B >> (j + 1))) break;
        std::vector<std::string> Q(half);
        for (int w2 = 0; w2 < half; ++w2) {
          Q[w2] = "P" + std::to_string(j) + "_" + std::to_string(w2);
          o << "    const float " << Q[w2] << " = " << P[2 * w2] << " + " << P[2 * w2 + 1] << ";\n";
        }
        P.swap(Q);
      }
      o << "    const float bb = bp * bp;\n";
      for (int i = 0; i < L; ++i) {
        const int b = run[i].bit, slot = run[i].slot;
        if (batched && slot >= 0) {
          const int pos = slot & 15;
          if (pend.tag[pos] >= 0 && pend.tag[pos] != slot) emit_flush(o, pend);
        }
        std::string g;
        if (b >= R)
          g = "flip_sign(" + P[0] + ", " + bit(b) + " << 31)";
        else if ((dirty >> b) & 1u)
          g = "flip_sign(gb" + std::to_string(b) + ", fs" + std::to_string(b) + ")";
        else
          g = "gb" + std::to_string(b);
        o << "    { float g = " << g << "; g *= gm" << i << " * bb;" << occ_scale(p, run[i].occ);
        if (slot < 0) {
          o << " (void)g;";
        } else if (batched) {
          const int pos = slot & 15;
          o << " pd" << pos << (pend.tag[pos] == slot ? " += g;" : " = g;")
            << " asm volatile(\"\" : \"+v\"(pd" << pos << "));";
          pend.tag[pos] = slot;
        } else if (gm.regs) {
          o << " const float gs = group_sum<" << gm.tm << ">(g); ga[" << slot / gm.tm
            << "] += (opaque(ln) == " << slot % gm.tm << "u) ? gs : 0.f; asm volatile(\"\" : \"+v\"(ga["
            << slot / gm.tm << "]));";
        } else {
          o << " { const float gs = group_sum<" << gm.tm << ">(g); if (w.leader) atomicAdd(&w.acc["
            << slot << " * w.G + w.grp], gs); }";
        }
        o << " }\n";
      }
    }
    for (int i = 0; i < L; ++i) o << "    bp *= tc" << i << ".y;\n";
    // The diagonal in double precision (every entry rounded to float once:
    // its rounding is shared by the amplitudes it multiplies, so a float
    // product's error, about sqrt(L) ulp, would shift the norm coherently).
    // The thread part: the product of 1 + i sg z over the thread-bit RZs.
    bool haveT = false;
    for (int i = 0; i < L; ++i) {
      if (run[i].bit < R) continue;
      const std::string x = std::string(sg) + "(double)z" + std::to_string(i);
      if (!haveT) {
        o << "    double Tr = 1.0, Ti = " << x << ";\n";
        haveT = true;
      } else {
        o << "    { const double x = " << x << ", nr = fma(-x, Ti, Tr); Ti = fma(x, Tr, Ti); Tr = nr; }\n";
      }
    }
    // per register bit: the factor for z = +1, 1 + i s (one RZ) or F (a
    // product); the factor for z = -1 is its conjugate
    std::vector<int> bits;
    std::map<int, int> cnt;
    for (int i = 0; i < L; ++i)
      if (run[i].bit < R && cnt[run[i].bit]++ == 0) bits.push_back(run[i].bit);
    std::sort(bits.begin(), bits.end());
    for (int b : bits) {
      bool first = true;
      for (int i = 0; i < L; ++i) {
        if (run[i].bit != b) continue;
        const std::string x = std::string(sg) + "(double)t" + std::to_string(i);
        if (cnt[b] == 1)
          o << "    const double s" << b << " = " << x << ";\n";
        else if (first)
          o << "    double F" << b << "r = 1.0, F" << b << "i = " << x << ";\n";
        else
          o << "    { const double x = " << x << ", nr = fma(-x, F" << b << "i, F" << b << "r); F"
            << b << "i = fma(x, F" << b << "r, F" << b << "i); F" << b << "r = nr; }\n";
        first = false;
      }
    }
    // y = x times bit b's factor for bit value h
    auto times = [&](const std::string& x, int b, int h, const std::string& y) {
      if (cnt[b] == 1) {
        const std::string sp = h ? "(-s" + std::to_string(b) + ")" : "s" + std::to_string(b);
        o << "const double " << y << "r = fma(-" << sp << ", " << x << "i, " << x << "r), " << y
          << "i = fma(" << sp << ", " << x << "r, " << x << "i);";
      } else {
        const std::string fr = "F" + std::to_string(b) + "r";
        const std::string fi = h ? "(-F" + std::to_string(b) + "i)" : "F" + std::to_string(b) + "i";
        o << "const double " << y << "r = fma(" << x << "r, " << fr << ", -(" << x << "i * " << fi
          << ")), " << y << "i = fma(" << x << "r, " << fi << ", " << x << "i * " << fr << ");";
      }
    };
    // the factor itself (the product's first factor when there is no thread part)
    auto first_factor = [&](int b, int h, const std::string& y) {
      if (cnt[b] == 1)
        o << "const double " << y << "r = 1.0, " << y << "i = " << (h ? "-" : "") << "s" << b << ";";
      else
        o << "const double " << y << "r = F" << b << "r, " << y << "i = " << (h ? "-" : "") << "F" << b
          << "i;";
    };
    auto apply = [&](int u, const char* st) {
      o << "      { const float xr = " << st << ".r[" << u << "], xi = " << st << ".i[" << u << "]; "
        << st << ".r[" << u << "] = fmaf(xr, er, -(xi * ei)); " << st << ".i[" << u
        << "] = fmaf(xr, ei, xi * er); }\n";
    };
    // depth-first over the register bits: one live product per level; at a
    // leaf (a value of every bit) the entry goes to float and multiplies the
    // amplitudes with those bits
    std::function<void(size_t, uint32_t, const std::string&)> walk =
        [&](size_t d, uint32_t val, const std::string& x) {
          if (d == bits.size()) {
            o << "    { const float er = (float)" << x << "r, ei = (float)" << x << "i;\n";
            uint32_t Bm = 0;
            for (int b : bits) Bm |= 1u << b;
            for (int u = 0; u < N; ++u) {
              if (((uint32_t)u & Bm) != val) continue;
              apply(u, "a");
              if (bwd) apply(u, "l");
            }
            o << "    }\n";
            return;
          }
          const int b = bits[d];
          for (int h = 0; h < 2; ++h) {
            const std::string y = "N" + std::to_string(d) + std::to_string(h);
            o << "    { ";
            if (x.empty()) first_factor(b, h, y);
            else times(x, b, h, y);
            o << "\n";
            walk(d + 1, val | ((uint32_t)h << b), y);
            o << "    }\n";
          }
        };
    walk(0, 0, haveT ? "T" : "");
    bool resc = false;
    for (int i = 0; i < L; ++i)
      if ((m + i) % kBlock == kBlock - 1 || m + i == nrot - 1) resc = true;
    m += L;
    if (resc) {
      o << "    rescale<R>(a, bp);";
      if (bwd) o << " rescale<R>(l, bp);";
      o << " bp = 1.f;\n";
    }
    o << "    gate_boundary(w);\n  }\n";
  };
  for (int pc = 0; pc < n_ins; ++pc) {
    const uint32_t w0 = ins[2 * pc], arg = ins[2 * pc + 1];
    const int op = w0 & 31, pa = (w0 >> 5) & 31, pb = (w0 >> 10) & 31;
    const int slot = (int)(w0 >> 16) - 1;
    switch (op) {
      case OP_EXCHANGE: {
        std::vector<std::pair<int, int>> swaps;
        if (lane_exchange(p, arg, k, R, t, swaps)) {
          // register bits swapped with lane bits: cross-lane moves, no LDS
          resolve(dirty);
          o << "  { const uint32_t ln = opaque(__lane_id());\n";
          for (const auto& sw : swaps) {
            o << "    lane_swap<R, " << sw.first << ", " << sw.second << ">(a, ln);\n";
            if (bwd) o << "    lane_swap<R, " << sw.first << ", " << sw.second << ">(l, ln);\n";
          }
          o << "  }\n";
          break;
        }
        o << "  { static constexpr uint32_t col[] = {";
        for (int i = 0; i < 2 * k; ++i) o << (i ? "," : "") << hex(p.cols[arg + i]);
        o << "};\n";
        // the swap frame, folded into the write addresses
        std::string fo = "0u";
        if (dirty) {
          o << "    const uint32_t fo = 0u";
          for (int r = 0; r < R; ++r)
            if ((dirty >> r) & 1u)
              o << " ^ ((col[" << r << "] << 2) & (uint32_t)((int32_t)fs" << r << " >> 31))";
          o << ";\n";
          fo = "fo";
        }
        if (bwd)
          o << "    exchange2<R>(a, l, w.xbuf, w.plane, col, " << k << ", " << t
            << ", w.stid, w.sl, " << fo << ");\n";
        else
          o << "    exchange<R>(a, w.xbuf, w.plane, col, " << k << ", " << t
            << ", w.stid, w.sl, " << fo << ");\n";
        for (int r = 0; r < R; ++r)
          if ((dirty >> r) & 1u) o << "    fs" << r << " = 0u;\n";
        dirty = 0;
        o << "  }\n";
        break;
      }
      case OP_CNOT: {
        const char* sts[2] = {"a", "l"};
        if (frames && pb < R && pa >= R) {
          // thread / tile control, register target: into the swap frame
          o << "  fs" << pb << " ^= " << bit(pa) << " << 31;\n";
          dirty |= 1u << pb;
          break;
        }
        if (pb >= R && pa < R) resolve(1u << pa);  // a register control of a lane target
        for (int s = 0; s < (bwd ? 2 : 1); ++s) {
          if (pb >= R && pa >= R + 2 && pa < R + 6)  // lane target, bank / row control
            o << "  cnot_ll<R, " << pb - R << ", " << pa - R << ">(" << sts[s] << ");\n";
          else if (pb >= R)  // target on a lane bit
            o << (pa < R ? "  cnot_rl<R, " + std::to_string(pa) + ", " + std::to_string(pb - R) +
                               ">(" + sts[s] + ");\n"
                         : "  cnot_tl<R, " + std::to_string(pb - R) + ">(" + sts[s] + ", " +
                               bit(pa) + ");\n");
          else if (pa < R)
            o << "  cnot_rr<R, " << pa << ", " << pb << ">(" << sts[s] << ");\n";
          else
            o << "  cnot_tr<R, " << pb << ">(" << sts[s] << ", " << bit(pa) << ");\n";
        }
        if (pa < R && pb < R && ((dirty >> pa) & 1u)) {
          // F CNOT(c, t) = CNOT(c, t) F X_t: the control's frame spreads to the target
          o << "  fs" << pb << " ^= fs" << pa << ";\n";
          dirty |= 1u << pb;
        }
        break;
      }
      case OP_CZ: {
        // A run of consecutive CZs is one diagonal of signs: amplitude u of the
        // thread is negated when c[u] ^ t0 ^ (XOR of m[r] over the register bits
        // r set in u) is 1.  c: the register/register pairs (compile time); m[r]:
        // the thread / tile bits paired with register bit r; t0: the products
        // of the thread / tile pairs.  One sign flip per value instead of one
        // per gate.
        int end = pc;
        while (end < n_ins && (ins[2 * end] & 31) == OP_CZ) ++end;
        {
          uint32_t regs = 0;
          for (int q = pc; q < end; ++q) {
            const int x = (ins[2 * q] >> 5) & 31, y = (ins[2 * q] >> 10) & 31;
            if (x < R) regs |= 1u << x;
            if (y < R) regs |= 1u << y;
          }
          resolve(regs);
        }
        const int N = 1 << R;
        std::vector<int> cu(N, 0);
        std::vector<std::string> mr(R);
        std::string t0;
        for (int q = pc; q < end; ++q) {
          const int x = (ins[2 * q] >> 5) & 31, y = (ins[2 * q] >> 10) & 31;
          const int lo = x < y ? x : y, hi = x < y ? y : x;
          if (hi < R) {
            for (int u = 0; u < N; ++u) cu[u] ^= (u >> lo) & (u >> hi) & 1;
          } else if (lo < R) {
            mr[lo] += (mr[lo].empty() ? "" : " ^ ") + std::string("(tb >> ") +
                      std::to_string(hi - R) + ")";
          } else {
            t0 += (t0.empty() ? "" : " ^ ") + std::string("((tb >> ") + std::to_string(lo - R) +
                  ") & (tb >> " + std::to_string(hi - R) + "))";
          }
        }
        o << "  { const uint32_t tb = opaque(w.tb); (void)tb;\n"
          << "    const uint32_t s0 = " << (t0.empty() ? "0u" : "(" + t0 + ") & 1u") << ";\n";
        for (int r = 0; r < R; ++r)
          o << "    const uint32_t m" << r << " = "
            << (mr[r].empty() ? "0u" : "(" + mr[r] + ") & 1u") << ";\n";
        for (int u = 1; u < N; ++u) {
          int low = 0;
          while (!((u >> low) & 1)) ++low;
          o << "    const uint32_t s" << u << " = s" << (u & (u - 1)) << " ^ m" << low << ";\n";
        }
        for (const char* st : {"a", "l"}) {
          if (st[0] == 'l' && !bwd) break;
          for (int u = 0; u < N; ++u)
            o << "    " << st << ".r[" << u << "] = flip_sign(" << st << ".r[" << u << "], (s" << u
              << " ^ " << cu[u] << "u) << 31); " << st << ".i[" << u << "] = flip_sign(" << st
              << ".i[" << u << "], (s" << u << " ^ " << cu[u] << "u) << 31);\n";
        }
        o << "  }\n";
        pc = end - 1;
        break;
      }
      default: {
        if (skip && (*skip)[arg]) break;  // a head rotation: run by the product start
        if (fuse && fusable_rz(p, w0, arg)) {
          std::vector<RzItem> run;
          int end = pc;
          for (; end < n_ins; ++end) {
            const uint32_t we = ins[2 * end], occ = ins[2 * end + 1];
            const int ope = we & 31;
            if (ope != OP_RX && ope != OP_RY && ope != OP_RZ) break;
            if (skip && (*skip)[occ]) continue;  // a head rotation: not run here
            if (!fusable_rz(p, we, occ)) break;
            run.push_back({(int)occ, (int)((ins[2 * end] >> 5) & 31), (int)(ins[2 * end] >> 16) - 1});
          }
          if (fused_cheaper(run)) {
            emit_rz_run(run);
            pc = end - 1;
            break;
          }
        }
        const bool reg = pa < R;
        const char* kind = op == OP_RX ? "rx" : op == OP_RY ? "ry" : "rz";
        if (batched && slot >= 0) {  // the slot's position is taken by another slot
          const int pos = slot & 15;
          if (pend.tag[pos] >= 0 && pend.tag[pos] != slot) emit_flush(o, pend);
        }
        const std::string at = std::to_string(arg) + " * " + std::to_string(S) + " + w.sl";
        if (tan) {
          if (sreg) {
            o << "  { const float2 tc = table_entry<" << arg % 64 << ">(T" << arg / 64 << "); ";
          } else if (ahead) {
            o << "  { const float2 tc = tcn; ";
            if (bwd) o << "const float gm = gmn; ";
            if (ri + 1 < rots.size()) {
              o << "tcn = w.tab[" << rots[ri + 1] << "]; ";
              if (bwd) o << "gmn = gmul[" << rots[ri + 1] << "]; ";
            }
            ++ri;
          } else {
            o << "  { const float2 tc = w.tab[" << arg << "]; ";
          }
          // negated under the swap frame (RY, RZ on a frame bit)
          const bool neg = reg && op != OP_RX && ((dirty >> pa) & 1u);
          if (neg)
            o << "const float t = flip_sign(tc.x, fs" << pa << "); ";
          else
            o << "const float t = tc.x; ";
          // RX / RY off the register bits sit on a lane bit (planner option)
          const std::string lane = std::to_string(pa - R);
          const std::string hi = pa >= R ? bit(pa) : "0u";
          if (!bwd) {
            if (reg)
              o << kind << "_t<R, " << pa << ">(a, t);";
            else if (op == OP_RZ)
              o << "phase_t<R>(a, flip_sign(t, " << hi << " << 31));";
            else if (op == OP_RX)
              o << "rx_lane_t<R, " << lane << ">(a, t);";
            else
              o << "ry_lane_t<R, " << lane << ">(a, t, " << hi << ");";
          } else {
            if (reg)
              o << "float g = adj_" << kind << "_t<R, " << pa << ">(a, l, t);";
            else if (op == OP_RZ)
              o << "float g = adj_phase_t<R>(a, l, t, " << hi << ");";
            else if (op == OP_RX)
              o << "float g = adj_rx_lane_t<R, " << lane << ">(a, l, t);";
            else
              o << "float g = adj_ry_lane_t<R, " << lane << ">(a, l, t, " << hi << ");";
            if (neg) o << " g = flip_sign(g, fs" << pa << ");";
            // the states carry 1 / (the factors of the block before this gate)
            if (sreg)
              o << " g *= table_entry<" << arg % 64 << ">(G" << arg / 64 << ") * (bp * bp);";
            else if (ahead)
              o << " g *= gm * (bp * bp);";
            else
              o << " g *= gmul[" << arg << "] * (bp * bp);";
            o << occ_scale(p, arg);
          }
          o << " bp *= tc.y;";
        } else {
          if (sreg)
            o << "  { const float2 cs = table_entry<" << arg % 64 << ">(T" << arg / 64 << "); ";
          else if (vreg)
            o << "  { const float2 cs = V" << arg << "; ";
          else
            o << "  { const float2 cs = w.tab[" << at << "]; ";
          // RX / RY off the register bits sit on a lane bit (planner option)
          const std::string lane = std::to_string(pa - R);
          const std::string hi = pa >= R ? bit(pa) : "0u";
          if (!bwd) {
            if (reg)
              o << kind << "_reg<R, " << pa << ">(a, cs.x, cs.y);";
            else if (op == OP_RZ)  // RZ on a thread / tile bit
              o << "phase_all<R>(a, cs.x, flip_sign(cs.y, (" << hi << " ^ 1u) << 31));";
            else if (op == OP_RX)
              o << "rx_lane<R, " << lane << ">(a, cs.x, cs.y);";
            else
              o << "ry_lane<R, " << lane << ">(a, cs.x, cs.y, " << hi << ");";
          } else {
            if (reg)
              o << "float g = adj_" << kind << "<R, " << pa << ">(a, l, cs.x, cs.y);";
            else if (op == OP_RZ)
              o << "float g = adj_rz_uniform<R>(a, l, cs.x, cs.y, " << hi << ");";
            else if (op == OP_RX)
              o << "float g = adj_rx_lane<R, " << lane << ">(a, l, cs.x, cs.y);";
            else
              o << "float g = adj_ry_lane<R, " << lane << ">(a, l, cs.x, cs.y, " << hi << ");";
            o << occ_scale(p, arg);
          }
        }
        if (bwd) {
          if (slot < 0) {
            o << " (void)g;";
          } else if (batched) {
            const int pos = slot & 15;
            // the empty asm keeps the partial's computation here: left free, the
            // compiler sinks it into the flush and keeps the old states alive
            o << " pd" << pos << (pend.tag[pos] == slot ? " += g;" : " = g;")
              << " asm volatile(\"\" : \"+v\"(pd" << pos << "));";
            pend.tag[pos] = slot;
          } else if (gm.regs)
            // the empty asm keeps the update here: left free, the additions drift
            // to the end of the kernel and every partial stays alive until then
            o << " const float gs = group_sum<" << gm.tm << ">(g); ga[" << slot / gm.tm
              << "] += (opaque(ln) == " << slot % gm.tm << "u) ? gs : 0.f; asm volatile(\"\" : \"+v\"(ga["
              << slot / gm.tm << "]));";
          else
            o << " { const float gs = group_sum<" << gm.tm << ">(g); if (w.leader) atomicAdd(&w.acc["
              << slot << " * w.G + w.grp], gs); }";
        }
        if (tan && (m % kBlock == kBlock - 1 || m == nrot - 1)) {
          o << " rescale<R>(a, bp);";
          if (bwd) o << " rescale<R>(l, bp);";
          o << " bp = 1.f;";
        }
        ++m;
        // gate by gate instruction selection (see gate_boundary); the small
        // kernels with gates on lane bits leave the scheduler free instead, so
        // that the DPP moves fold into the multiplies that use them
        o << (p.lanes > 0 ? " }\n" : " gate_boundary(w); }\n");
      }
    }
  }
  if (batched) emit_flush(o, pend);
  if (frames) {
    if (fend == kFrameResolve) resolve(dirty);
    for (int r = 0; r < R; ++r) o << "  (void)fs" << r << ";\n";
  }
}

// The circuit's constants, compiled in (the interpreter reads them from the
// plan's arrays): the qubit count, the mapping (qubit -> physical bit) that
// the <Z> epilogue or the forming of lambda uses (map_off in the plan's maps),
// and every angle occurrence's record.  A gate list's constants then cost no
// dependent loads from device memory before the first gate.
void emit_constants(std::ostringstream& o, const Plan& p, int map_off) {
  o << "static constexpr int kN = " << p.n << ", kNocc = " << p.occ_src.size()
    << ", kS = " << (p.path == VQC_PATH_RESIDENT ? p.S : 1) << ";\n"
    << "__device__ __forceinline__ static uint32_t zmask(const uint8_t*, const uint32_t*, "
       "int q) {\n";
  // physical bits of each measured qubit's Z-string under this mapping
  std::vector<uint32_t> zm(p.n);
  for (int q = 0; q < p.n; ++q) {
    const uint32_t m = p.zmask.empty() ? 1u << q : p.zmask[q];
    uint32_t pm = 0;
    for (int b = 0; b < p.n; ++b)
      if ((m >> b) & 1u) pm |= 1u << p.maps[map_off + b];
    zm[q] = pm;
  }
  emit_array(o, "uint32_t", "t", zm);
  o << "  return t[q];\n}\n"
    << "__device__ __forceinline__ static OccRec occ(const int32_t*, const int32_t*, const float*, "
       "const float*, int o) {\n";
  // The records as runs of occurrences with one source and (a, b) whose index
  // grows by one (parameters and inputs read in order, as most ansatz layers
  // do) or stays (one parameter shared by a layer): a few compares instead of
  // a load from the code object's data, whose latency would come before the
  // first parameter load.  Circuits with many runs (constant gates each make
  // one) use the table.
  const int nocc = (int)p.occ_src.size();
  auto rec_a = [&](int i) {
    return p.occ_src[i] == kSrcConst ? p.occ_cs[2 * i] : p.affine ? p.occ_ma[2 * i] : 1.f;
  };
  auto rec_b = [&](int i) {
    return p.occ_src[i] == kSrcConst ? p.occ_cs[2 * i + 1] : p.affine ? p.occ_ma[2 * i + 1] : 0.f;
  };
  std::vector<int> starts, stride;
  for (int i = 0; i < nocc; ++i) {
    bool cont = i > 0 && p.occ_src[i] != kSrcConst && p.occ_src[i] == p.occ_src[i - 1] &&
                rec_a(i) == rec_a(i - 1) && rec_b(i) == rec_b(i - 1);
    const int d = i > 0 ? p.occ_idx[i] - p.occ_idx[i - 1] : -1;
    if (cont && i - 1 == starts.back()) {  // the run's second member sets its stride
      cont = d == 0 || d == 1;
      if (cont) stride.back() = d;
    } else if (cont) {
      cont = d == stride.back();
    }
    if (!cont) {
      starts.push_back(i);
      stride.push_back(1);
    }
  }
  constexpr size_t kMaxRuns = 16;
  o << std::hexfloat;
  if (nocc > 0 && starts.size() <= kMaxRuns) {
    o << "  OccRec r;\n";
    for (size_t j = 0; j < starts.size(); ++j) {
      const int i = starts[j];
      const int end = j + 1 < starts.size() ? starts[j + 1] : nocc;
      o << "  " << (j ? "else " : "") << (j + 1 < starts.size() ? "if (o < " +
                                                                  std::to_string(end) + ") " : "")
        << "r = OccRec{" << p.occ_src[i] << ", "
        << (stride[j] ? "o + " + std::to_string(p.occ_idx[i] - i) : std::to_string(p.occ_idx[i]))
        << ", " << (double)rec_a(i) << "f, " << (double)rec_b(i) << "f};\n";
    }
    o << "  return r;\n}\n";
  } else {
    o << "  static constexpr OccRec t[] = {";
    for (int i = 0; i < nocc; ++i)
      o << (i ? ", " : "") << "{" << p.occ_src[i] << ", " << p.occ_idx[i] << ", "
        << (double)rec_a(i) << "f, " << (double)rec_b(i) << "f}";
    if (nocc == 0) o << "{0, 0, 0.f, 0.f}";
    o << "};\n  return t[o];\n}\n";
  }
  o << std::defaultfloat;
}

// A schedule struct: run() for one stream, the group sum used for <Z>, and
// (when `tables`) the kernel's tangent-form tables.
void emit_sched_struct(std::ostringstream& o, const std::string& name, const Plan& p,
                       const uint32_t* ins, int n_ins, bool bwd, int R, int k, int S,
                       const GradMode& gm, const TanMode& tm, const Frame* tables, int map_off,
                       bool load = false, int fixed_flags = -1,
                       const std::vector<char>* skip = nullptr,
                       const std::string& head = std::string(), FrameEnd fend = kFrameResolve) {
  o << "struct " << name << " {\n";
  emit_constants(o, p, map_off);
  o << "static constexpr int kFixedFlags = " << fixed_flags << ";\n";
  // the streaming step's product head (stream_product_start, stream_head_partials)
  if (head.empty()) o << "static constexpr bool kProductStart = false, kHeadPartials = false;\n";
  else o << head;
  o
    << "template <int R, bool BWD, bool WIDE>\n"
    << "__device__ __forceinline__ static void run(St<R>& a, St<R>& l, const Walk& w, "
       "const uint32_t*, int) {\n"
    << "  (void)l;\n";
  const bool regs = bwd && gm.regs && gm.nr > 0;
  if (regs)
    o << "  const uint32_t ln = (uint32_t)w.stid & " << gm.tm - 1 << "u;\n"
      << "  float ga[" << gm.nr << "];\n"
      << "#pragma unroll\n  for (int j = 0; j < " << gm.nr << "; ++j) ga[j] = 0.f;\n";
  emit_schedule(o, p, ins, n_ins, bwd, R, k, S, gm, tm, skip, fend);
  if (regs)  // every (slot, group) accumulator is written by exactly one lane
    o << "#pragma unroll\n  for (int j = 0; j < " << gm.nr << "; ++j) {\n"
      << "    const uint32_t slot = j * " << gm.tm << "u + "
      << (batched_flush(p, bwd, gm, R, k) ? "((ln & 3u) | ((ln >> 2) & 12u) | ((ln << 2) & 48u))"
                                          : "ln")
      << ";\n"
      << "    if (slot < " << gm.ns << "u) w.acc[slot * w.G + w.grp] = ga[j];\n  }\n";
  o << "}\n"
    << "__device__ __forceinline__ static float lane_sum(float v, const Walk&) {\n"
    << "  return group_sum<" << gm.tm << ">(v);\n}\n";
  if (tables) emit_tables(o, p, tm, *tables, S << (k - R), false, load, skip);
  o << "};\n";
}

size_t lds_size(size_t b) { return b < 16 ? 16 : b; }

// Kernels holding 16 amplitudes per thread ask for three waves per SIMD (at
// most 168 VGPRs, a few spilled to scratch): left free, the compiler gave the
// 12-qubit training step 178 VGPRs and two waves, and the 14-qubit forward
// passes 178-184.  Measured: 12-qubit step 1.37 -> 1.05 ms, 14-qubit step
// 13.5 -> 12.9 ms; four waves (128 VGPRs) spill too much (14.2 ms).  The
// 32-amplitude adjoint passes gained nothing from it.
std::string occupancy(int R) {
  return R == 4 ? "__attribute__((amdgpu_waves_per_eu(3))) " : "";
}

// Whether a kernel uses the tangent form: one sample per workgroup (the frame
// is per sample).  With 4 amplitudes per thread the tables are read from
// registers (table_row), and rotations on lane bits take the lane forms
// (rx_lane_t, ...).
bool tangent_wanted(int S, int R) {
  (void)R;
  return S == 1;
}

// One kernel in a program of its own, so that the kernels of a circuit compile
// in parallel.  esign: the kernel computes <Z> (forward) or forms lambda
// (adjoint).
std::string kernel_unit(const Plan& p, const Frame& fr, const std::string& name,
                        const uint32_t* ins, int n_ins, bool bwd, bool stream, int R, int S,
                        int threads, size_t lds, int n_slots, bool esign, int map_off,
                        bool load = false, int fixed_flags = -1,
                        const std::string& head = std::string()) {
  std::ostringstream o;
  o << "#include \"vqc_device.h\"\nnamespace vqc {\n";
  const int lanes = stream ? threads : 1 << (p.k - R);
  TanMode tm = tan_mode(p, bwd ? nullptr : ins, n_ins, bwd ? ins : nullptr, n_ins, S, esign, lds);
  tm.on = tm.on && tangent_wanted(S, R);
  // the swap frame at the stream's end: resolved where the state is read or
  // stored after the sweep, dropped by a resident adjoint and by the last
  // streaming adjoint pass without a product head (nothing reads their states)
  FrameEnd fend = bwd ? kFrameDrop : kFrameResolve;
  if (stream && bwd && (!(fixed_flags & PF_LAST_ADJ) || !head.empty())) fend = kFrameResolve;
  emit_sched_struct(o, "Sched", p, ins, n_ins, bwd, R, p.k, S, grad_mode(lanes, n_slots), tm, &fr,
                    map_off, load, fixed_flags, nullptr, head, fend);
  o << "}  // namespace vqc\n"
    << "extern \"C\" __global__ void __launch_bounds__(" << threads << ") " << occupancy(R)
    << name
    << (stream ? "(const vqc::PassArgs A) {\n" : "(const vqc::TileArgs A) {\n")
    << "  __shared__ __align__(16) unsigned char smem[" << lds_size(tm.on ? tm.end : lds) << "];\n";
  if (stream)
    o << "  vqc::stream_body<" << (bwd ? "true" : "false") << ", " << R << ", " << p.k
      << ", vqc::Sched>(A, smem);\n}\n";
  else
    o << "  vqc::resident_body<" << threads << ", " << (bwd ? "true" : "false") << ", " << R
      << ", vqc::Sched>(A, smem);\n}\n";
  return o.str();
}

// The product head of the training step (vqc_device.h, "product head"): the
// occurrences of the head rotations (per occurrence, 1 for a head rotation),
// or an empty vector when the step runs every rotation.  Needs the tangent
// form's one sample per workgroup, one lane per qubit and 16-bit occurrence
// and slot numbers.
std::vector<char> head_occurrences(const Plan& p, const TanMode& tm) {
  std::vector<char> h;
  if (!tm.on || p.S != 1 || p.n > 64 || p.head.empty()) return h;
  const size_t nocc = p.occ_src.size();
  bool any = false;
  for (const auto& hq : p.head)
    for (const Prim& g : hq) {
      if (g.occ >= 65536 || p.occ_slot[g.occ] >= 65535) return {};
      any = true;
    }
  if (!any) return h;
  h.assign(nocc, 0);
  for (const auto& hq : p.head)
    for (const Prim& g : hq) h[g.occ] = 1;
  return h;
}

// Longest head.
int head_len(const Plan& p) {
  int L = 0;
  for (const auto& hq : p.head) L = std::max(L, (int)hq.size());
  return L;
}

// kL and fn(tid): lane q's head steps (HeadPre: word = occurrence | kind << 16,
// gradient slot + 1, chain-rule factor), lanes >= n clamped to qubit n - 1.
void emit_head_pre(std::ostringstream& o, const Plan& p, const char* fn) {
  const int L = head_len(p), n = p.n;
  o << "static constexpr int kL = " << L << ";\n";
  std::vector<uint32_t> words, slots;
  std::vector<float> muls;
  bool scaled = false;
  for (int q = 0; q < n; ++q)
    for (int i = 0; i < L; ++i) {
      if (i < (int)p.head[q].size()) {
        const Prim& g = p.head[q][i];
        const uint32_t kind = g.kind == P_RX ? 0u : g.kind == P_RY ? 1u : 2u;
        words.push_back((uint32_t)g.occ | kind << 16);
        slots.push_back((uint32_t)(p.occ_slot[g.occ] + 1));
        const float m = p.affine ? p.occ_ma[2 * g.occ] : 1.f;
        muls.push_back(m);
        scaled = scaled || m != 1.f;
      } else {
        words.push_back(3u << 16);
        slots.push_back(0u);
        muls.push_back(1.f);
      }
    }
  o << "__device__ __forceinline__ static HeadPre<kL> " << fn << "(int tid) {\n";
  emit_array(o, "uint32_t", "kW", words);
  emit_array(o, "uint32_t", "kS", slots);
  if (scaled) {
    o << "  static constexpr float kM[] = {";
    for (size_t i = 0; i < muls.size(); ++i)
      o << (i ? "," : "") << std::hexfloat << (double)muls[i] << "f" << std::defaultfloat;
    o << "};\n";
  }
  o << "  const int q = min(tid & 63, " << n - 1 << ");\n"
    << "  HeadPre<kL> h;\n"
    << "#pragma unroll\n"
    << "  for (int i = 0; i < kL; ++i) {\n"
    << "    h.w[i] = kW[q * kL + i];\n"
    << "    h.s[i] = (int32_t)kS[q * kL + i];\n"
    << "    h.m[i] = " << (scaled ? "kM[q * kL + i]" : "1.f") << ";\n"
    << "  }\n"
    << "  return h;\n}\n";
}

// The qubits on the register bits (reg, R of them) and on the bits of w.tb
// (tb: thread bits, then a streaming tile's index bits) under the mapping at
// map_off; -1 where no qubit sits (tile ranks >= nq of a small state).
void head_bits(const Plan& p, int map_off, int R, int ntb, std::vector<int>& reg,
               std::vector<int>& tb) {
  reg.assign(R, -1);
  tb.assign(ntb, -1);
  for (int q = 0; q < p.nq; ++q) {
    const int ph = p.maps[map_off + q];
    if (ph < R) reg[ph] = q;
    else if (ph - R < ntb) tb[ph - R] = q;
  }
}

// const float2 a<q>, b<q>: qubit q's head state from lane q (after head_walk
// or head_state left it in fa, fb); qubits >= n stay |0>.
void emit_head_broadcast(std::ostringstream& o, const Plan& p) {
  for (int q = 0; q < p.n; ++q)
    o << "  const float2 a" << q << " = make_float2(lane_value(fa.x, " << q << "), lane_value(fa.y, "
      << q << ")), b" << q << " = make_float2(lane_value(fb.x, " << q << "), lane_value(fb.y, " << q
      << "));\n";
  for (int q = p.n; q < std::max(p.nq, p.k); ++q)
    o << "  const float2 a" << q << " = make_float2(1.f, 0.f), b" << q
      << " = make_float2(0.f, 0.f);\n";
}

// The product state's amplitudes in a: the factors of the tb bits, then one
// doubling per register bit.
void emit_product_state(std::ostringstream& o, const std::vector<int>& reg,
                        const std::vector<int>& tbq) {
  const int R = (int)reg.size();
  o << "  const uint32_t tb = w.tb;\n"
    << "  float2 t = make_float2(1.f, 0.f);\n";
  for (size_t j = 0; j < tbq.size(); ++j)
    if (tbq[j] >= 0)
      o << "  t = cmul(t, ((tb >> " << j << ") & 1u) ? b" << tbq[j] << " : a" << tbq[j] << ");\n";
  o << "  const float2 A0_0 = t;\n";
  for (int pb = 0; pb < R; ++pb)
    for (int u = 0; u < (2 << pb); ++u) {
      const int src = u & ~(1 << pb);
      o << "  const float2 A" << pb + 1 << "_" << u << " = cmul(A" << pb << "_" << src << ", "
        << (((u >> pb) & 1) ? "b" : "a") << reg[pb] << ");\n";
    }
  for (int u = 0; u < (1 << R); ++u)
    o << "  a.r[" << u << "] = A" << R << "_" << u << ".x; a.i[" << u << "] = A" << R << "_" << u
      << ".y;\n";
}

// float v[NV]: this thread's terms of v_q = (I_q (x) <phi_{not q}|) lambda for
// every qubit q < n (v[4 q .. 4 q + 3] = v_q(0), v_q(1) as re, im), from
// lambda in l under the mapping given by reg / tbq; a<q>, b<q> in scope.
void emit_head_contraction(std::ostringstream& o, const Plan& p, const std::vector<int>& reg,
                           const std::vector<int>& tbq, int NV) {
  const int R = (int)reg.size(), t = (int)tbq.size(), n = p.n;
  o << "  const uint32_t tb = w.tb;\n";
  // the tb bits' factors, and their products leaving one out
  for (int j = 0; j < t; ++j)
    o << "  const float2 f" << j << " = ((tb >> " << j << ") & 1u) ? b" << tbq[j] << " : a"
      << tbq[j] << ";\n";
  o << "  const float2 P0 = make_float2(1.f, 0.f);\n";
  for (int j = 0; j < t; ++j)
    o << "  const float2 P" << j + 1 << " = cmul(P" << j << ", f" << j << ");\n";
  if (t > 0) o << "  const float2 S" << t - 1 << " = make_float2(1.f, 0.f);\n";
  for (int j = t - 2; j >= 0; --j)
    o << "  const float2 S" << j << " = cmul(S" << j + 1 << ", f" << j + 1 << ");\n";
  for (int j = 0; j < t; ++j)
    o << "  const float2 T" << j << " = cmul(P" << j << ", S" << j << ");\n";
  o << "  const float2 tall = P" << t << ";\n";
  for (int u = 0; u < (1 << R); ++u)
    o << "  const float2 x" << u << " = make_float2(l.r[" << u << "], l.i[" << u << "]);\n";
  // for each register bit: lambda contracted over the other register bits
  for (int pb = 0; pb < R; ++pb) {
    std::vector<std::string> name(1 << R);
    for (int u = 0; u < (1 << R); ++u) name[u] = "x" + std::to_string(u);
    int done = 0;
    for (int c = R - 1; c >= 0; --c) {
      if (c == pb) continue;
      for (int u = 0; u < (1 << R); ++u) {
        if (((u >> c) & 1) || (u & done)) continue;
        const std::string nm = "y" + std::to_string(pb) + "_" + std::to_string(c) + "_" +
                               std::to_string(u);
        o << "  const float2 " << nm << " = cadd(cmulc(a" << reg[c] << ", " << name[u]
          << "), cmulc(b" << reg[c] << ", " << name[u | (1 << c)] << "));\n";
        name[u] = nm;
      }
      done |= 1 << c;
    }
    o << "  const float2 C" << pb << "_0 = " << name[0] << ", C" << pb << "_1 = " << name[1 << pb]
      << ";\n";
  }
  o << "  const float2 sall = cadd(cmulc(a" << reg[0] << ", C0_0), cmulc(b" << reg[0]
    << ", C0_1));\n"
    << "  float v[" << NV << "];\n"
    << "#pragma unroll\n  for (int j = 0; j < " << NV << "; ++j) v[j] = 0.f;\n";
  for (int pb = 0; pb < R; ++pb) {
    const int q = reg[pb];
    if (q >= n) continue;
    o << "  { const float2 u0 = cmulc(tall, C" << pb << "_0), u1 = cmulc(tall, C" << pb << "_1);\n"
      << "    v[" << 4 * q << "] = u0.x; v[" << 4 * q + 1 << "] = u0.y; v[" << 4 * q + 2
      << "] = u1.x; v[" << 4 * q + 3 << "] = u1.y; }\n";
  }
  for (int j = 0; j < t; ++j) {
    const int q = tbq[j];
    if (q >= n) continue;
    o << "  { const float2 c = cmulc(T" << j << ", sall); const bool one = (tb >> " << j
      << ") & 1u;\n"
      << "    v[" << 4 * q << "] = one ? 0.f : c.x; v[" << 4 * q + 1 << "] = one ? 0.f : c.y; v["
      << 4 * q + 2 << "] = one ? c.x : 0.f; v[" << 4 * q + 3 << "] = one ? c.y : 0.f; }\n";
  }
}

int head_nv(const Plan& p) { return (4 * p.n + 15) / 16 * 16; }

// struct Head of the training step: the head tables and mappings.
void emit_head(std::ostringstream& o, const Plan& p, size_t off) {
  const int L = head_len(p), n = p.n, k = p.k, R = p.R;
  o << "struct Head {\n"
    << "static constexpr bool kOn = true;\n"
    << "static constexpr int kN = " << n << ", kK = " << k << ";\n"
    << "static constexpr uint32_t kOff = " << off << "u;\n";
  emit_head_pre(o, p, "preload");
  o << "using Pre = HeadPre<kL>;\n";
  std::vector<int> sreg, sthr, ereg, ethr;
  head_bits(p, p.start_off, R, k - R, sreg, sthr);
  head_bits(p, p.bwd_end_off, R, k - R, ereg, ethr);
  // init(): every head walked by its qubit's lane, then the product state in
  // the forward's start mapping
  o << "template <int R>\n"
    << "__device__ __forceinline__ static void init(St<R>& a, const Walk& w, const Pre& hp) {\n"
    << "  static_assert(R == " << R << ", \"register width\");\n"
    << "  HeadRec* rec = reinterpret_cast<HeadRec*>(w.smem + kOff);\n"
    << "  float4* fin = reinterpret_cast<float4*>(w.smem + kOff + " << n * L * 32 << "u);\n"
    << "  float2 fa, fb;\n"
    << "  head_walk<kL>(w, hp, rec, fin, kN, fa, fb);\n";
  emit_head_broadcast(o, p);
  emit_product_state(o, sreg, sthr);
  o << "}\n";
  // grads(): the 2-vector partials of every qubit from lambda in the adjoint's
  // end mapping, then the sums and the walks back (head_finish)
  const int NV = head_nv(p);
  o << "template <int WG, int R>\n"
    << "__device__ __forceinline__ static void grads(const St<R>& l, const Walk& w) {\n"
    << "  const HeadRec* rec = reinterpret_cast<const HeadRec*>(w.smem + kOff);\n"
    << "  const float4* fin = reinterpret_cast<const float4*>(w.smem + kOff + " << n * L * 32
    << "u);\n";
  for (int q = 0; q < n; ++q)
    o << "  const float4 F" << q << " = fin[" << q << "];\n"
      << "  const float2 a" << q << " = make_float2(F" << q << ".x, F" << q << ".y), b" << q
      << " = make_float2(F" << q << ".z, F" << q << ".w);\n";
  for (int q = n; q < k; ++q)
    o << "  const float2 a" << q << " = make_float2(1.f, 0.f), b" << q
      << " = make_float2(0.f, 0.f);\n";
  emit_head_contraction(o, p, ereg, ethr, NV);
  o << "  head_finish<WG, kL, " << NV << ">(v, w, rec, kN);\n"
    << "}\n"
    << "};\n";
}

// The streaming training step's first forward pass: product_start() builds the
// state after the heads in the pass's start mapping (map_off).
std::string stream_product_start(const Plan& p, int map_off, int R) {
  std::ostringstream o;
  std::vector<int> reg, tbq;
  head_bits(p, map_off, R, p.k - R + p.ng, reg, tbq);
  o << "static constexpr bool kProductStart = true, kHeadPartials = false;\n";
  emit_head_pre(o, p, "head_pre");
  o << "template <int R>\n"
    << "__device__ __forceinline__ static void product_start(St<R>& a, const Walk& w) {\n"
    << "  static_assert(R == " << R << ", \"register width\");\n"
    << "  const HeadPre<kL> hp = head_pre((int)threadIdx.x);\n"
    << "  float2 fa, fb;\n"
    << "  head_state<kL>(w, hp, fa, fb);\n";
  emit_head_broadcast(o, p);
  emit_product_state(o, reg, tbq);
  o << "}\n";
  return o.str();
}

// The streaming training step's last adjoint pass: head_partials() sums this
// tile's terms of every v_q over the workgroup and stores them to out[0, NV).
std::string stream_head_partials(const Plan& p, int map_off, int R) {
  std::ostringstream o;
  std::vector<int> reg, tbq;
  head_bits(p, map_off, R, p.k - R + p.ng, reg, tbq);
  const int NV = head_nv(p);
  o << "static constexpr bool kProductStart = false, kHeadPartials = true;\n"
    << "static constexpr int kNV = " << NV << ";\n";
  emit_head_pre(o, p, "head_pre");
  o << "template <int WG, int R>\n"
    << "__device__ __forceinline__ static void head_partials(const St<R>& l, const Walk& w, "
       "float* out) {\n"
    << "  static_assert(R == " << R << ", \"register width\");\n"
    << "  const HeadPre<kL> hp = head_pre((int)threadIdx.x);\n"
    << "  float2 fa, fb;\n"
    << "  head_state<kL>(w, hp, fa, fb);\n";
  emit_head_broadcast(o, p);
  emit_head_contraction(o, p, reg, tbq, NV);
  o << "  const float s = workgroup_sums<WG, " << NV << ">(v, w.xbuf);\n"
    << "  if ((int)threadIdx.x < " << NV << ") out[threadIdx.x] = s;\n"
    << "}\n";
  return o.str();
}

// The streaming training step's head gradient kernel (head_finish_stream): its
// Head struct holds the head tables and, per gradient slot of a head rotation,
// the list of its (qubit, step) terms.
std::string head_finish_unit(const Plan& p, const std::string& name) {
  std::ostringstream o;
  const int L = head_len(p), n = p.n, NV = head_nv(p);
  const int NS = p.P + p.F;
  o << "#include \"vqc_device.h\"\nnamespace vqc {\nstruct Head {\n"
    << "static constexpr int kN = " << n << ", kNV = " << NV << ", kNS = " << NS
    << ", kNG = " << p.ng << ";\n";
  emit_head_pre(o, p, "head_pre");
  std::map<int, std::vector<int>> terms;  // slot -> q * L + i
  for (int q = 0; q < n; ++q)
    for (int i = 0; i < (int)p.head[q].size(); ++i) {
      const int s = p.occ_slot[p.head[q][i].occ];
      if (s >= 0) terms[s].push_back(q * L + i);
    }
  std::vector<uint32_t> start{0}, idx, slot;
  bool unique = true;  // no two head rotations share a gradient slot
  for (const auto& kv : terms) {
    slot.push_back((uint32_t)kv.first);
    idx.insert(idx.end(), kv.second.begin(), kv.second.end());
    start.push_back((uint32_t)idx.size());
    unique = unique && kv.second.size() == 1;
  }
  o << "static constexpr bool kUniqueSlots = " << (unique ? "true" : "false") << ";\n";
  o << "__device__ __forceinline__ static void add_grads(const float* gs, float* hs, int tid, "
       "int nt) {\n";
  emit_array(o, "uint32_t", "kStart", start);
  emit_array(o, "uint32_t", "kIdx", idx);
  emit_array(o, "uint32_t", "kSlot", slot);
  o << "  for (int i = tid; i < " << slot.size() << "; i += nt) {\n"
    << "    float s = 0.f;\n"
    << "    for (uint32_t e = kStart[i]; e < kStart[i + 1]; ++e) s += gs[kIdx[e]];\n"
    << "    hs[kSlot[i]] = s;\n"
    << "  }\n}\n"
    << "};\n}  // namespace vqc\n";
  const size_t lds = (size_t)n * L * 32 + (size_t)n * 16 + (size_t)(NV + n * L + NS) * 4;
  o << "extern \"C\" __global__ void __launch_bounds__(" << kHeadThreads << ") " << name
    << "(const vqc::PassArgs A) {\n"
    << "  __shared__ __align__(16) unsigned char smem[" << lds_size(lds) << "];\n"
    << "  vqc::head_finish_stream<" << kHeadThreads << ", vqc::Head>(A, smem);\n}\n";
  return o.str();
}

// The training step: forward and adjoint sweeps in one kernel.
std::string step_unit(const Plan& p, const Frame& fr) {
  std::ostringstream o;
  o << "#include \"vqc_device.h\"\nnamespace vqc {\n";
  const int lanes = 1 << (p.k - p.R);
  const GradMode gm = grad_mode(lanes, p.P + p.F);
  const int nf = (int)p.fwd.size() / 2, nb = (int)p.bwd.size() / 2;
  TanMode tm = tan_mode(p, p.fwd.data(), nf, p.bwd.data(), nb, p.S, true, p.lds_step);
  tm.on = tm.on && tangent_wanted(p.S, p.R);
  std::vector<char> head = head_occurrences(p, tm);
  size_t head_off = 0, end = tm.on ? tm.end : p.lds_step;
  if (!head.empty()) {
    int L = 0;
    for (const auto& hq : p.head) L = std::max(L, (int)hq.size());
    head_off = align16(end);
    const size_t head_end = head_off + (size_t)p.n * L * 32 + (size_t)p.n * 16;
    if (head_end <= (size_t)kLdsBytes) {
      end = head_end;
      // the sweeps' own rotations (the tables' signs and the block rescales)
      auto drop = [&](std::vector<int>& v) {
        v.erase(std::remove_if(v.begin(), v.end(), [&](int occ) { return head[occ] != 0; }),
                v.end());
      };
      drop(tm.focc);
      drop(tm.bocc);
    } else {
      head.clear();
    }
  }
  const std::vector<char>* skip = head.empty() ? nullptr : &head;
  emit_sched_struct(o, "SchedF", p, p.fwd.data(), nf, false, p.R, p.k, p.S, gm, tm, &fr,
                    p.end_off, false, -1, skip, std::string(), kFrameResolve);
  emit_sched_struct(o, "SchedB", p, p.bwd.data(), nb, true, p.R, p.k, p.S, gm, tm, nullptr,
                    p.end_off, false, -1, skip, std::string(),
                    skip ? kFrameResolve : kFrameDrop);
  if (skip) emit_head(o, p, head_off);
  o << "}  // namespace vqc\n"
    << "extern \"C\" __global__ void __launch_bounds__(" << p.WG << ") " << occupancy(p.R)
    << "vqc_rs(const vqc::TileArgs A) {\n"
    << "  __shared__ __align__(16) unsigned char smem[" << lds_size(end) << "];\n"
    << "  vqc::resident_step_body<" << p.WG << ", " << p.R << ", vqc::SchedF, vqc::SchedB"
    << (skip ? ", vqc::Head" : "") << ">(A, smem);\n}\n";
  return o.str();
}

}  // namespace

// The table kernel of a streaming circuit: the angle table and the frame signs
// of every occurrence, per sample (table_body), or "" when they do not fit in
// LDS (the passes then compute their own).
// With a product head the head rotations keep their exact (cos, sin) and
// take no part in the frame.
std::string table_unit(const Plan& p, const Frame& fr, const std::string& name = "vqc_st") {
  TanMode t;
  const int nocc = (int)p.occ_src.size();
  t.W = std::max(1, (nocc + 31) / 32);
  std::vector<char> head;
  if (p.product_head) {
    head.assign(nocc, 0);
    for (const auto& hq : p.head)
      for (const Prim& g : hq) head[g.occ] = 1;
  }
  for (int k = 0; k < nocc; ++k)
    if (head.empty() || !head[k]) t.focc.push_back(k);
  t.esign = true;
  size_t off = align16((size_t)std::max(nocc, 1) * 8);
  t.off_bits = off;
  off = align16(off + (size_t)(t.W + 1) * 4);
  t.off_gm = off;
  off = align16(off + (size_t)std::max(nocc, 1) * 4);
  t.off_es = off;
  off = align16(off + (size_t)p.n * 4);
  t.end = off;
  t.on = nocc > 0 && t.end <= (size_t)kLdsBytes;
  if (!t.on) return "";
  std::ostringstream o;
  o << "#include \"vqc_device.h\"\nnamespace vqc {\nstruct Sched {\n";
  emit_constants(o, p, p.end_off);
  emit_tables(o, p, t, fr, kTableThreads, true, false, head.empty() ? nullptr : &head);
  o << "};\n}  // namespace vqc\n"
    << "extern \"C\" __global__ void __launch_bounds__(" << kTableThreads
    << ") " << name << "(const vqc::PassArgs A) {\n"
    << "  __shared__ __align__(16) unsigned char smem[" << t.end << "];\n"
    << "  vqc::table_body<" << kTableThreads << ", vqc::Sched>(A, smem);\n}\n";
  return o.str();
}

std::vector<JitUnit> jit_units(const Plan& p) {
  std::vector<JitUnit> u;
  const Frame fr = frame_rows(p);
  if (p.path == VQC_PATH_RESIDENT) {
    u.push_back({"vqc_rf", kernel_unit(p, fr, "vqc_rf", p.fwd.data(), (int)p.fwd.size() / 2,
                                       false, false, p.R, p.S, p.WG, p.lds_fwd, p.P + p.F, true,
                                       p.end_off), 'r'});
    u.push_back({"vqc_rb", kernel_unit(p, fr, "vqc_rb", p.bwd.data(), (int)p.bwd.size() / 2,
                                       true, false, p.R, p.S, p.WG, p.lds_bwd, p.P + p.F, true,
                                       p.end_off), 'b'});
    u.push_back({"vqc_rs", step_unit(p, fr), 's'});
    return u;
  }
  // the training step's plan with a product head: vqc_hf* / vqc_hb* / vqc_ht /
  // vqc_hg, apart in traces from the whole circuit's vqc_sf* / vqc_sb* / vqc_st
  const std::string pre = p.product_head ? "vqc_h" : "vqc_s";
  const std::string tables = table_unit(p, fr, pre + "t");
  const bool load = !tables.empty();
  const bool ph = p.product_head && load;  // the heads' exact angles come from the tables
  for (size_t i = 0; i < p.fpass.size(); ++i) {
    const std::string name = pre + "f" + std::to_string(i);
    const PassPlan& pp = p.fpass[i];
    const std::string head = ph && (pp.flags & PF_INIT)
                                 ? stream_product_start(p, pp.start_off, p.Rf) : std::string();
    u.push_back({name, kernel_unit(p, fr, name, p.fwd.data() + 2 * pp.ins_off, pp.n_ins, false,
                                   true, p.Rf, 1, 1 << (p.k - p.Rf), p.lds_fwd, pp.n_slots,
                                   (pp.flags & PF_ZPART) != 0, pp.end_off, load,
                                   (int)(pp.flags & ~PF_INIT), head), 'F'});
  }
  for (size_t i = 0; i < p.bpass.size(); ++i) {
    const std::string name = pre + "b" + std::to_string(i);
    const PassPlan& pp = p.bpass[i];
    const std::string head = ph && (pp.flags & PF_LAST_ADJ)
                                 ? stream_head_partials(p, pp.end_off, p.Rb) : std::string();
    u.push_back({name, kernel_unit(p, fr, name, p.bwd.data() + 2 * pp.ins_off, pp.n_ins, true,
                                   true, p.Rb, 1, 1 << (p.k - p.Rb), p.lds_bwd, pp.n_slots,
                                   (pp.flags & PF_MAKE_LAMBDA) != 0, pp.start_off, load,
                                   (int)(pp.flags & ~PF_INIT), head), 'B'});
  }
  if (load) u.push_back({pre + "t", tables, 'T'});
  if (ph) u.push_back({"vqc_hg", head_finish_unit(p, "vqc_hg"), 'G'});
  return u;
}

// Whether a streaming plan's passes read their tables from the table kernel
// (which a product head needs).
bool stream_tables_fit(const Plan& p) {
  return !table_unit(p, frame_rows(p)).empty();
}

namespace {

// The helper next to this library (vqc_jitc), or "" when it is missing.
const std::string& helper_path() {
  static const std::string path = [] {
    Dl_info info;
    if (dladdr(reinterpret_cast<void*>(&compile_source), &info) && info.dli_fname) {
      const std::string lib = info.dli_fname;
      const size_t slash = lib.rfind('/');
      const std::string h = (slash == std::string::npos ? std::string(".") : lib.substr(0, slash)) +
                            "/vqc_jitc";
      if (access(h.c_str(), X_OK) == 0) return h;
    }
    return std::string();
  }();
  return path;
}

bool read_file(const std::string& path, std::vector<char>& out) {
  FILE* f = std::fopen(path.c_str(), "rb");
  if (!f) return false;
  out.clear();
  char buf[1 << 16];
  size_t n;
  while ((n = std::fread(buf, 1, sizeof buf, f)) > 0) out.insert(out.end(), buf, buf + n);
  std::fclose(f);
  return true;
}

bool write_file(const std::string& path, const std::string& text) {
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f) return false;
  const bool ok = std::fwrite(text.data(), 1, text.size(), f) == text.size();
  return std::fclose(f) == 0 && ok;
}

// Compiles the sources in child processes of the helper, at most `slots` at a
// time.  Returns false when the helper could not be run (the caller then
// compiles in this process); a failed compilation returns true with rc set.
bool compile_in_children(const std::vector<const std::string*>& srcs, size_t slots,
                         std::vector<std::vector<char>>& codes, int& rc, std::string& log) {
  const std::string& helper = helper_path();
  if (helper.empty()) return false;
  const char* tmp = std::getenv("TMPDIR");
  std::string dir = std::string(tmp && *tmp ? tmp : "/tmp") + "/vqcjit.XXXXXX";
  if (!mkdtemp(&dir[0])) return false;
  const size_t n = srcs.size();
  std::vector<std::string> in(n), out(n), err(n);
  bool ok = true;
  for (size_t i = 0; i < n && ok; ++i) {
    in[i] = dir + "/k" + std::to_string(i) + ".hip";
    out[i] = dir + "/k" + std::to_string(i) + ".co";
    err[i] = dir + "/k" + std::to_string(i) + ".log";
    ok = write_file(in[i], *srcs[i]);
  }
  std::vector<int> status(n, -1);
  std::vector<pid_t> pid(n, -1);
  size_t next = 0, running = 0, done = 0;
  while (ok && done < n) {
    while (next < n && running < slots) {
      posix_spawn_file_actions_t fa;
      posix_spawn_file_actions_init(&fa);
      posix_spawn_file_actions_addopen(&fa, 2, err[next].c_str(), O_WRONLY | O_CREAT | O_TRUNC,
                                       0644);
      char* argv[] = {const_cast<char*>(helper.c_str()), const_cast<char*>(in[next].c_str()),
                      const_cast<char*>(out[next].c_str()), nullptr};
      const int e = posix_spawn(&pid[next], helper.c_str(), &fa, nullptr, argv, environ);
      posix_spawn_file_actions_destroy(&fa);
      if (e != 0) {
        ok = false;
        break;
      }
      ++next;
      ++running;
    }
    bool reaped = false;
    for (size_t i = 0; i < next; ++i) {
      if (pid[i] <= 0 || status[i] != -1) continue;
      int st = 0;
      const pid_t r = waitpid(pid[i], &st, WNOHANG);
      if (r == pid[i] || r < 0) {
        status[i] = (r == pid[i] && WIFEXITED(st)) ? WEXITSTATUS(st) : 255;
        --running;
        ++done;
        reaped = true;
      }
    }
    if (!reaped && ok) usleep(2000);
  }
  // children still running after a spawn failure are waited for
  for (size_t i = 0; i < next; ++i)
    if (pid[i] > 0 && status[i] == -1) {
      int st = 0;
      (void)waitpid(pid[i], &st, 0);
      status[i] = 255;
    }
  rc = VQC_OK;
  if (ok) {
    codes.assign(n, {});
    for (size_t i = 0; i < n; ++i) {
      if (status[i] == 0 && read_file(out[i], codes[i])) continue;
      if (status[i] == 1) {  // the compiler rejected the source
        std::vector<char> text;
        read_file(err[i], text);
        log.assign(text.begin(), text.end());
        rc = VQC_ERR_UNSUPPORTED;
      } else {
        ok = false;  // the helper itself failed: compile here instead
      }
      break;
    }
  }
  for (size_t i = 0; i < n; ++i) {
    unlink(in[i].c_str());
    unlink(out[i].c_str());
    unlink(err[i].c_str());
  }
  rmdir(dir.c_str());
  return ok;
}

// Compiles every source; returns the first failure.  Several kernels go to
// helper processes in parallel (VQC_JIT_INPROC=1 keeps everything in this
// process, where compilations run one at a time).
int compile_all(const std::vector<const std::string*>& srcs, std::vector<std::vector<char>>& codes,
                std::string& log) {
  const unsigned hw = std::thread::hardware_concurrency();
  const size_t slots = std::min<size_t>(srcs.size(), hw ? std::min(hw, 16u) : 4u);
  const char* inproc = std::getenv("VQC_JIT_INPROC");
  if (slots > 1 && !(inproc && *inproc == '1')) {
    int rc = VQC_OK;
    if (compile_in_children(srcs, slots, codes, rc, log)) return rc;
  }
  codes.assign(srcs.size(), {});
  for (size_t i = 0; i < srcs.size(); ++i) {
    const int rc = compile_source(*srcs[i], codes[i], log);
    if (rc != VQC_OK) return rc;
  }
  return VQC_OK;
}

// VQC_JIT_DUMP=<directory>: write each generated kernel to <directory>/<name>.hip
void dump_units(const std::vector<JitUnit>& units) {
  const char* dir = std::getenv("VQC_JIT_DUMP");
  if (!dir || !*dir) return;
  for (const JitUnit& u : units) {
    const std::string path = std::string(dir) + "/" + u.name + ".hip";
    if (FILE* f = std::fopen(path.c_str(), "w")) {
      std::fwrite(u.src.data(), 1, u.src.size(), f);
      std::fclose(f);
    }
  }
}

std::mutex g_cache_mu;
// (device, kernel source) -> function; the modules stay loaded until exit
std::map<std::string, hipFunction_t> g_cache;

}  // namespace

int jit_compile_only(const Plan& p, std::string& log) {
  const std::vector<JitUnit> units = jit_units(p);
  dump_units(units);
  std::vector<const std::string*> srcs;
  for (const JitUnit& u : units) srcs.push_back(&u.src);
  std::vector<std::vector<char>> codes;
  return compile_all(srcs, codes, log);
}

int jit_build(const Plan& p, int device, JitKernels& out, std::string& msg) {
  const std::vector<JitUnit> units = jit_units(p);
  dump_units(units);
  const std::string dev = std::to_string(device) + "\n";
  std::vector<hipFunction_t> fns(units.size(), nullptr);
  std::vector<size_t> missing;
  {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    for (size_t i = 0; i < units.size(); ++i) {
      auto it = g_cache.find(dev + units[i].src);
      if (it != g_cache.end()) fns[i] = it->second;
      else missing.push_back(i);
    }
  }
  if (!missing.empty()) {
    std::vector<const std::string*> srcs;
    for (size_t i : missing) srcs.push_back(&units[i].src);
    std::vector<std::vector<char>> codes;
    std::string log;
    if (compile_all(srcs, codes, log) != VQC_OK) {
      msg = "run-time compilation of the circuit kernels failed: " + log.substr(0, 4000);
      return VQC_ERR_UNSUPPORTED;
    }
    std::lock_guard<std::mutex> lock(g_cache_mu);
    for (size_t j = 0; j < missing.size(); ++j) {
      const size_t i = missing[j];
      const std::string key = dev + units[i].src;
      auto it = g_cache.find(key);
      if (it != g_cache.end()) {  // a concurrent compile won
        fns[i] = it->second;
        continue;
      }
      hipModule_t mod = nullptr;
      if (hipModuleLoadData(&mod, codes[j].data()) != hipSuccess) {
        msg = "hipModuleLoadData failed for " + units[i].name;
        return VQC_ERR_HIP;
      }
      if (hipModuleGetFunction(&fns[i], mod, units[i].name.c_str()) != hipSuccess) {
        msg = "hipModuleGetFunction failed for " + units[i].name;
        return VQC_ERR_HIP;
      }
      g_cache[key] = fns[i];
    }
  }
  out = JitKernels();
  for (size_t i = 0; i < units.size(); ++i) {
    switch (units[i].role) {
      case 'r': out.res_fwd = fns[i]; break;
      case 'b': out.res_bwd = fns[i]; break;
      case 's': out.res_step = fns[i]; break;
      case 'T': out.tables = fns[i]; break;
      case 'G': out.head_finish = fns[i]; break;
      case 'F': out.pass_fwd.push_back(fns[i]); break;
      case 'B': out.pass_bwd.push_back(fns[i]); break;
      default: break;
    }
  }
  return VQC_OK;
}

int jit_launch(void* fn, int64_t blocks, int threads, const void* args, size_t args_size,
               void* stream) {
  (void)args_size;
  void* params[] = {const_cast<void*>(args)};
  return (int)hipModuleLaunchKernel((hipFunction_t)fn, (unsigned)blocks, 1, 1, (unsigned)threads,
                                    1, 1, 0, (hipStream_t)stream, params, nullptr);
}

}  // namespace vqc
