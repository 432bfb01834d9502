// host_harness.cpp -- the host-only code of the library (compile-phase
// validation and lowering, stream / register-tile planning, kernel source
// generation, the OpenQASM front end and the C ABI's argument checks) driven
// by seeded random and malformed inputs, for a build with AddressSanitizer and
// UndefinedBehaviorSanitizer (tests/test_sanitize_cpu.py).  No device is used:
// every circuit is compiled with device = -1, and the device launchers the
// ABI links against are stubs that abort if reached.
//
//   host_harness <seed> <circuits> <qasm mutations>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <string>
#include <vector>

#include "vqc.h"
#include "vqc_internal.h"

// ------------------------------------------------- device stubs (never called)
namespace vqc {
[[noreturn]] static void no_device(const char* what) {
  std::fprintf(stderr, "host harness reached device code: %s\n", what);
  std::abort();
}
int launch_resident_forward(const Plan&, const TileArgs&, int64_t, void*) { no_device("fwd"); }
int launch_resident_backward(const Plan&, const TileArgs&, int64_t, void*) { no_device("bwd"); }
int launch_resident_step(const Plan&, const TileArgs&, int64_t, void*) { no_device("step"); }
int launch_stream_pass(const Plan&, bool, const PassArgs&, int64_t, void*) { no_device("pass"); }
int launch_reduce_e(int64_t, int, int, const float*, float*, void*) { no_device("reduce_e"); }
int launch_reduce_e_loss(int64_t, int, int, const float*, float*, int, int64_t, const float*,
                         float*, void*) {
  no_device("reduce_e_loss");
}
int launch_reduce_grad(int64_t, int, int, int, int, const float*, float*, float*, void*) {
  no_device("reduce_grad");
}
int launch_fill_zero(float*, int64_t, void*) { no_device("fill"); }
int launch_fd_combine(int64_t, int, int, int, int, int, float, const float*, const float*, float*,
                      float*, void*) {
  no_device("fd");
}
int launch_sum_rows(int64_t, int, const float*, float*, void*) { no_device("sum_rows"); }
int launch_loss_grad(int, int64_t, int64_t, int, const float*, const float*, float*, void*) {
  no_device("loss");
}
int prepare_kernels(const Plan&) { no_device("prepare"); }
int scratch_pointer(int, void**) { no_device("scratch"); }
}  // namespace vqc

// ------------------------------------------------- seeded generator (splitmix64)
struct Rng {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  int below(int n) { return n <= 0 ? 0 : (int)(next() % (uint64_t)n); }
  float unit() { return (float)(next() >> 40) / (float)(1ull << 24); }
};

static int g_fail = 0;
#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++g_fail;                                                              \
    }                                                                        \
  } while (0)

static bool is_status(int rc) { return rc == VQC_OK || (rc <= -1 && rc >= -6); }

// A random gate record; with `bad` some fields go out of range.
static vqc_op random_op(Rng& r, int n, int P, int F, bool bad) {
  vqc_op o;
  std::memset(&o, 0, sizeof(o));
  o.kind = bad && r.below(20) == 0 ? r.below(40) - 4 : r.below(32);
  for (int w = 0; w < 3; ++w) o.wires[w] = bad && r.below(25) == 0 ? r.below(n + 3) - 1 : r.below(n);
  for (int s = 0; s < 3; ++s) {
    o.src[s] = bad && r.below(30) == 0 ? r.below(5) - 1 : r.below(3);
    const int lim = o.src[s] == VQC_SRC_PARAM ? P : F;
    o.idx[s] = bad && r.below(30) == 0 ? r.below(lim + 3) - 1 : r.below(lim > 0 ? lim : 1);
    o.val[s] = (r.unit() - 0.5f) * 8.f;
    o.mul[s] = r.below(4) == 0 ? (r.unit() - 0.5f) * 4.f : 1.f;
    if (bad && r.below(40) == 0) o.val[s] = std::numeric_limits<float>::quiet_NaN();
    if (bad && r.below(40) == 0) o.mul[s] = 0.f;
    if (bad && r.below(60) == 0) o.mul[s] = std::numeric_limits<float>::infinity();
  }
  return o;
}

static void circuits(Rng& r, int count) {
  for (int it = 0; it < count; ++it) {
    const bool bad = r.below(3) == 0;
    const int n = 1 + r.below(it % 7 == 0 ? 20 : 16);
    const int P = r.below(40), F = r.below(n + 2);
    const int n_ops = r.below(it % 11 == 0 ? 400 : 90);
    std::vector<vqc_op> ops;
    for (int i = 0; i < n_ops; ++i) ops.push_back(random_op(r, n, P, F, bad));
    vqc_compile_opts opts;
    std::memset(&opts, 0, sizeof(opts));
    opts.device = -1;
    opts.path = r.below(5) == 0 ? r.below(4) : 0;
    opts.reg_bits = r.below(4) == 0 ? r.below(7) : 0;
    opts.engine = r.below(6) == 0 ? r.below(3) : 0;
    opts.shared_params = r.below(5) == 0 ? r.below(3) : 0;
    const int tiles[] = {0, 0, 0, 12, 13, 14, 15};
    opts.tile_qubits = tiles[r.below(7)];
    if (bad && r.below(20) == 0) opts.reserved[r.below(2)] = 1;
    vqc_circuit* c = nullptr;
    const int rc = vqc_compile(ops.data(), (int32_t)ops.size(), n, P, F, &opts, &c);
    CHECK(is_status(rc));
    CHECK((rc == VQC_OK) == (c != nullptr));
    if (rc != VQC_OK) {
      CHECK(std::strlen(vqc_last_error()) > 0);
      continue;
    }
    vqc_info info;
    CHECK(vqc_circuit_info(c, &info) == VQC_OK);
    CHECK(info.n_qubits == n && info.n_params == P && info.n_inputs == F);
    for (int mode = -1; mode <= 4; ++mode)
      for (int64_t b : {(int64_t)-1, (int64_t)0, (int64_t)1, (int64_t)37, (int64_t)4096}) {
        const size_t nb = vqc_workspace_bytes(c, b, mode);
        CHECK((nb == (size_t)-1) == (b < 0 || mode < 0 || mode > 3));
      }
    // a host-only handle cannot run: every entry point refuses before any HIP call
    float dummy[4] = {0, 0, 0, 0};
    CHECK(vqc_forward(c, 1, dummy, dummy, dummy, nullptr, 0, nullptr) == VQC_ERR_INVALID_ARG);
    CHECK(vqc_backward(c, 1, dummy, dummy, dummy, nullptr, 0, dummy, dummy, nullptr) ==
          VQC_ERR_INVALID_ARG);
    CHECK(vqc_train_step(c, 1, dummy, dummy, 0, nullptr, dummy, nullptr, nullptr, nullptr,
                         nullptr, 0, nullptr) == VQC_ERR_INVALID_ARG);
    CHECK(vqc_train_step_noalloc(c, 1, dummy, dummy, 0, nullptr, dummy, nullptr, nullptr,
                                 nullptr, nullptr) == VQC_ERR_INVALID_ARG);
    CHECK(vqc_fd_backward(c, 1, dummy, dummy, dummy, 0.1f, nullptr, 0, dummy, dummy, nullptr) ==
          VQC_ERR_INVALID_ARG);
    vqc_destroy(c);
    // the kernel generator over the same plan (source text only, no compiler)
    if (opts.engine == VQC_ENGINE_JIT && it % 3 == 0) {
      std::vector<vqc::HostOp> hops(ops.size());
      for (size_t i = 0; i < ops.size(); ++i) {
        hops[i].kind = ops[i].kind;
        for (int s = 0; s < 3; ++s) {
          hops[i].w[s] = ops[i].wires[s];
          hops[i].src[s] = ops[i].src[s];
          hops[i].idx[s] = ops[i].idx[s];
          hops[i].val[s] = ops[i].val[s];
          hops[i].mul[s] = ops[i].mul[s];
        }
      }
      vqc::Plan p;
      std::string msg;
      if (vqc::build_plan(hops, n, P, F, opts.path, opts.reg_bits, p, msg, true,
                          opts.tile_qubits) == 0) {
        const std::vector<vqc::JitUnit> units = vqc::jit_units(p);
        CHECK(!units.empty());
        for (const vqc::JitUnit& u : units) CHECK(u.src.find("__global__") != std::string::npos);
      }
    }
  }
}

// ------------------------------------------------- OpenQASM corpus and mutations
static const char* const kGates1[] = {"h", "x", "y", "z", "s", "sdg", "t", "tdg", "sx", "id"};
static const char* const kGates1p[] = {"rx", "ry", "rz", "p", "u1"};
static const char* const kGates2[] = {"cx", "cz", "cy", "ch", "swap"};
static const char* const kGates2p[] = {"crx", "cry", "crz", "cp", "rxx", "ryy", "rzz"};

static std::string angle(Rng& r) {
  switch (r.below(6)) {
    case 0: return "pi/" + std::to_string(1 + r.below(8));
    case 1: return "theta[" + std::to_string(r.below(4)) + "]";
    case 2: return "2*x[" + std::to_string(r.below(3)) + "] + 0.5";
    case 3: return "-(pi - theta[1])/3";
    case 4: return "sin(0.3)*x[0]";
    default: return std::to_string(r.unit() * 6.0f - 3.0f);
  }
}

static std::string program(Rng& r, bool& v3) {
  const int n = 2 + r.below(6);
  v3 = r.below(2) != 0;
  std::string s = v3 ? "OPENQASM 3.0;\ninclude \"stdgates.inc\";\n"
                     : "OPENQASM 2.0;\ninclude \"qelib1.inc\";\n";
  if (v3) {
    s += "qubit[" + std::to_string(n) + "] q;\nbit[" + std::to_string(n) + "] c;\n";
    s += "input array[float[64], 4] theta;\ninput array[float[32], 3] x;\n";
  } else {
    s += "qreg q[" + std::to_string(n) + "];\ncreg c[" + std::to_string(n) + "];\n";
  }
  s += "gate g2(a) u, v { rz(a) u; cx u, v; ry(-a/2) v; }\n";
  const int lines = 3 + r.below(14);
  for (int i = 0; i < lines; ++i) {
    const int a = r.below(n), b = (a + 1 + r.below(n - 1)) % n;
    const std::string qa = "q[" + std::to_string(a) + "]", qb = "q[" + std::to_string(b) + "]";
    switch (r.below(7)) {
      case 0: s += std::string(kGates1[r.below(10)]) + " " + qa + ";\n"; break;
      case 1: s += std::string(kGates1p[r.below(5)]) + "(" + (v3 ? angle(r) : "pi/3") + ") " + qa + ";\n"; break;
      case 2: s += std::string(kGates2[r.below(5)]) + " " + qa + ", " + qb + ";\n"; break;
      case 3: s += std::string(kGates2p[r.below(7)]) + "(" + (v3 ? angle(r) : "0.25") + ") " + qa + ", " + qb + ";\n"; break;
      case 4: s += "u3(0.1, " + std::string(v3 ? angle(r) : "0.2") + ", 0.3) " + qa + ";\n"; break;
      case 5: s += "g2(" + std::string(v3 ? angle(r) : "pi") + ") " + qa + ", " + qb + ";\n"; break;
      default: s += "barrier q;\n"; break;
    }
  }
  s += v3 ? "c = measure q;\n" : "measure q -> c;\n";
  return s;
}

static std::string mutate(Rng& r, std::string s) {
  static const char* const tokens[] = {";", "(", ")", "[", "]", "{", "}", ",", "->", "pi", "q",
                                       "gate", "if", "reset q[0];", "measure", "*", "/", "^",
                                       "-", "1e999", "0x", "\"", "//", "/*", "\n", "input",
                                       "float[64]", "qubit[0] z;", "cx q[0], q[0];"};
  const int k = 1 + r.below(4);
  for (int i = 0; i < k && !s.empty(); ++i) {
    const size_t pos = (size_t)r.below((int)s.size());
    switch (r.below(5)) {
      case 0: s.erase(pos, 1 + r.below(6)); break;
      case 1: s.insert(pos, tokens[r.below((int)(sizeof(tokens) / sizeof(tokens[0])))]); break;
      case 2: s[pos] = (char)(32 + r.below(95)); break;
      case 3: s.resize(pos); break;
      default: s[pos] = (char)r.below(256); break;  // arbitrary bytes, NUL excluded below
    }
  }
  for (char& ch : s)
    if (ch == '\0') ch = ' ';
  return s;
}

static void qasm(Rng& r, int count) {
  for (int it = 0; it < count; ++it) {
    bool v3 = false;
    std::string src = program(r, v3);
    const bool mutated = it % 4 != 0;
    if (mutated) src = mutate(r, src);
    int32_t n_ops = 0, nq = 0, P = 0, F = 0;
    const char* names = v3 && r.below(2) ? "x" : nullptr;  // only v3 programs declare x
    int rc = vqc_parse_qasm(src.c_str(), names, nullptr, 0, &n_ops, &nq, &P, &F);
    CHECK(is_status(rc));
    if (!mutated) CHECK(rc == VQC_OK);
    if (rc == VQC_OK) {
      std::vector<vqc_op> ops((size_t)n_ops + 1);
      rc = vqc_parse_qasm(src.c_str(), names, ops.data(), n_ops, &n_ops, &nq, &P, &F);
      CHECK(rc == VQC_OK);
      if (n_ops > 0) {  // one gate too few is refused
        rc = vqc_parse_qasm(src.c_str(), names, ops.data(), n_ops - 1, &n_ops, &nq, &P, &F);
        CHECK(rc == VQC_ERR_TOO_LARGE);
      }
      vqc_compile_opts opts;
      std::memset(&opts, 0, sizeof(opts));
      opts.device = -1;
      vqc_circuit* c = nullptr;
      rc = vqc_compile_qasm(src.c_str(), names, &opts, &c);
      CHECK(is_status(rc));
      vqc_destroy(c);
    } else {
      CHECK(std::strlen(vqc_last_error()) > 0);
    }
  }
  // degenerate inputs
  int32_t a = 0, b = 0, c = 0, d = 0;
  CHECK(vqc_parse_qasm("", nullptr, nullptr, 0, &a, &b, &c, &d) != VQC_OK);
  CHECK(vqc_parse_qasm(nullptr, nullptr, nullptr, 0, &a, &b, &c, &d) != VQC_OK);
  CHECK(vqc_parse_qasm("OPENQASM 2.0;", nullptr, nullptr, 0, nullptr, &b, &c, &d) ==
        VQC_ERR_INVALID_ARG);
  std::string deep = "OPENQASM 2.0;\ninclude \"qelib1.inc\";\nqreg q[1];\n";
  for (int i = 0; i < 200; ++i) deep += "gate h" + std::to_string(i + 1) + " a { h" +
                                        (i ? std::to_string(i) : std::string("")) + " a; }\n";
  deep += "h200 q[0];\n";
  CHECK(is_status(vqc_parse_qasm(deep.c_str(), nullptr, nullptr, 0, &a, &b, &c, &d)));
  std::string nest = "OPENQASM 3.0;\nqubit q;\nrx(";
  for (int i = 0; i < 5000; ++i) nest += "(";
  nest += "1";
  for (int i = 0; i < 5000; ++i) nest += ")";
  nest += ") q;\n";
  CHECK(is_status(vqc_parse_qasm(nest.c_str(), nullptr, nullptr, 0, &a, &b, &c, &d)));
}

int main(int argc, char** argv) {
  const uint64_t seed = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 1;
  const int nc = argc > 2 ? std::atoi(argv[2]) : 300;
  const int nq = argc > 3 ? std::atoi(argv[3]) : 2000;
  Rng r{seed};
  circuits(r, nc);
  qasm(r, nq);
  std::printf("host harness: seed %llu, %d circuits, %d programs, %d failures\n",
              (unsigned long long)seed, nc, nq, g_fail);
  return g_fail ? 1 : 0;
}
