// jit.cpp -- compile once: the circuit's schedule becomes straight-line gfx950
// code (Sec. 3 "Compile-Once Lowering and Execution").
//
// The planner's instruction streams are turned into source text in which every
// register position, exchange layout and gradient slot is a literal: a gate is a
// call of the register-tile template for its position, a CNOT between register
// bits is a renaming, and exchanges use constant column tables.  The text plus
// the shared device code (vqc_device.h) is compiled with hiprtc for gfx950, one
// program per kernel on a pool of host threads, and loaded as modules; launches
// go through hipModuleLaunchKernel.  Identical kernels are compiled once per
// process.
#include <hip/hip_runtime_api.h>
#include <hip/hiprtc.h>

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

namespace vqc {

// Shared headers embedded at build time (generated from vqc.h, vqc_structs.h,
// vqc_device.h).
extern const int kJitHeaderCount;
extern const char* const kJitHeaderNames[];
extern const char* const kJitHeaderSources[];

namespace {

std::string hex(uint32_t v) {
  char b[16];
  std::snprintf(b, sizeof b, "0x%xu", v);
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

// Statements of one instruction stream for register width R.
void emit_schedule(std::ostringstream& o, const Plan& p, const uint32_t* ins, int n_ins, bool bwd,
                   int R, int k, int S, const GradMode& gm) {
  const int t = k - R;
  for (int pc = 0; pc < n_ins; ++pc) {
    const uint32_t w0 = ins[2 * pc], arg = ins[2 * pc + 1];
    const int op = w0 & 31, pa = (w0 >> 5) & 31, pb = (w0 >> 10) & 31;
    const int slot = (int)(w0 >> 16) - 1;
    switch (op) {
      case OP_EXCHANGE: {
        o << "  { static constexpr uint32_t col[] = {";
        for (int i = 0; i < 2 * k; ++i) o << (i ? "," : "") << hex(p.cols[arg + i]);
        o << "};\n    exchange<R>(a, w.xbuf, w.plane, col, " << k << ", " << t
          << ", w.stid, w.sl);\n";
        if (bwd)
          o << "    exchange<R>(l, w.xbuf, w.plane, col, " << k << ", " << t
            << ", w.stid, w.sl);\n";
        o << "  }\n";
        break;
      }
      case OP_CNOT: {
        const char* sts[2] = {"a", "l"};
        for (int s = 0; s < (bwd ? 2 : 1); ++s) {
          if (pa < R)
            o << "  cnot_rr<R, " << pa << ", " << pb << ">(" << sts[s] << ");\n";
          else
            o << "  cnot_tr<R, " << pb << ">(" << sts[s] << ", tile_bit<R>(w, " << pa << "));\n";
        }
        break;
      }
      case OP_CZ: {
        const int lo = pa < pb ? pa : pb, hi = pa < pb ? pb : pa;
        for (const char* st : {"a", "l"}) {
          if (st[0] == 'l' && !bwd) break;
          if (hi < R)
            o << "  cz_rr<R, " << lo << ", " << hi << ">(" << st << ");\n";
          else if (lo < R)
            o << "  cz_tr<R, " << lo << ">(" << st << ", tile_bit<R>(w, " << hi << "));\n";
          else
            o << "  negate_if<R>(" << st << ", tile_bit<R>(w, " << lo << ") & tile_bit<R>(w, "
              << hi << "));\n";
        }
        break;
      }
      default: {
        o << "  { const float2 cs = w.tab[" << arg << " * " << S << " + w.sl]; ";
        const bool reg = pa < R;
        const char* kind = op == OP_RX ? "rx" : op == OP_RY ? "ry" : "rz";
        if (!bwd) {
          if (reg)
            o << kind << "_reg<R, " << pa << ">(a, cs.x, cs.y);";
          else  // RZ on a thread / tile bit
            o << "phase_all<R>(a, cs.x, flip_sign(cs.y, (tile_bit<R>(w, " << pa
              << ") ^ 1u) << 31));";
        } else {
          if (reg)
            o << "const float g = adj_" << kind << "<R, " << pa << ">(a, l, cs.x, cs.y);";
          else
            o << "const float g = adj_rz_uniform<R>(a, l, cs.x, cs.y, tile_bit<R>(w, " << pa
              << "));";
          if (slot < 0)
            o << " (void)g;";
          else if (gm.regs)
            // the empty asm keeps the update here: left free, the additions drift
            // to the end of the kernel and every partial stays alive until then
            o << " const float gs = group_sum<" << gm.tm << ">(g); ga[" << slot / gm.tm
              << "] += (opaque(ln) == " << slot % gm.tm << "u) ? gs : 0.f; asm volatile(\"\" : \"+v\"(ga["
              << slot / gm.tm << "]));";
          else
            o << " { const float gs = group_sum<" << gm.tm << ">(g); if (w.leader) atomicAdd(&w.acc["
              << slot << " * w.G + w.grp], gs); }";
        }
        o << " gate_boundary(w); }\n";
      }
    }
  }
}

void emit_sched_struct(std::ostringstream& o, const std::string& name, const Plan& p,
                       const uint32_t* ins, int n_ins, bool bwd, int R, int k, int S,
                       const GradMode& gm) {
  o << "struct " << name << " {\n"
    << "template <int R, bool BWD, bool WIDE>\n"
    << "__device__ __forceinline__ static void run(St<R>& a, St<R>& l, const Walk& w, "
       "const uint32_t*, int) {\n"
    << "  (void)l;\n";
  const bool regs = bwd && gm.regs && gm.nr > 0;
  if (regs)
    o << "  const uint32_t ln = (uint32_t)w.stid & " << gm.tm - 1 << "u;\n"
      << "  float ga[" << gm.nr << "];\n"
      << "#pragma unroll\n  for (int j = 0; j < " << gm.nr << "; ++j) ga[j] = 0.f;\n";
  emit_schedule(o, p, ins, n_ins, bwd, R, k, S, gm);
  if (regs)  // every (slot, group) accumulator is written by exactly one lane
    o << "#pragma unroll\n  for (int j = 0; j < " << gm.nr << "; ++j) {\n"
      << "    const uint32_t slot = j * " << gm.tm << "u + ln;\n"
      << "    if (slot < " << gm.ns << "u) w.acc[slot * w.G + w.grp] = ga[j];\n  }\n";
  o << "}\n"
    << "__device__ __forceinline__ static float lane_sum(float v, const Walk&) {\n"
    << "  return group_sum<" << gm.tm << ">(v);\n}\n};\n";
}

size_t lds_size(size_t b) { return b < 16 ? 16 : b; }

// One kernel in a program of its own, so that the kernels of a circuit compile
// in parallel.
std::string kernel_unit(const Plan& p, const std::string& name, const uint32_t* ins, int n_ins,
                        bool bwd, bool stream, int R, int S, int threads, size_t lds,
                        int n_slots) {
  std::ostringstream o;
  o << "#include \"vqc_device.h\"\nnamespace vqc {\n";
  const int lanes = stream ? threads : 1 << (p.k - R);
  emit_sched_struct(o, "Sched", p, ins, n_ins, bwd, R, p.k, S, grad_mode(lanes, n_slots));
  o << "}  // namespace vqc\n"
    << "extern \"C\" __global__ void __launch_bounds__(" << threads << ") " << name
    << (stream ? "(const vqc::PassArgs A) {\n" : "(const vqc::TileArgs A) {\n")
    << "  __shared__ __align__(16) unsigned char smem[" << lds_size(lds) << "];\n";
  if (stream)
    o << "  vqc::stream_body<" << (bwd ? "true" : "false") << ", " << R
      << ", vqc::Sched>(A, smem);\n}\n";
  else
    o << "  vqc::resident_body<" << threads << ", " << (bwd ? "true" : "false") << ", " << R
      << ", vqc::Sched>(A, smem);\n}\n";
  return o.str();
}

}  // namespace

std::vector<JitUnit> jit_units(const Plan& p) {
  std::vector<JitUnit> u;
  if (p.path == VQC_PATH_RESIDENT) {
    u.push_back({"vqc_rf", kernel_unit(p, "vqc_rf", p.fwd.data(), (int)p.fwd.size() / 2, false,
                                       false, p.R, p.S, p.WG, p.lds_fwd, p.P + p.F)});
    u.push_back({"vqc_rb", kernel_unit(p, "vqc_rb", p.bwd.data(), (int)p.bwd.size() / 2, true,
                                       false, p.R, p.S, p.WG, p.lds_bwd, p.P + p.F)});
    return u;
  }
  for (size_t i = 0; i < p.fpass.size(); ++i) {
    const std::string name = "vqc_sf" + std::to_string(i);
    u.push_back({name, kernel_unit(p, name, p.fwd.data() + 2 * p.fpass[i].ins_off,
                                   p.fpass[i].n_ins, false, true, p.Rf, 1, 1 << (p.k - p.Rf),
                                   p.lds_fwd, p.fpass[i].n_slots)});
  }
  for (size_t i = 0; i < p.bpass.size(); ++i) {
    const std::string name = "vqc_sb" + std::to_string(i);
    u.push_back({name, kernel_unit(p, name, p.bwd.data() + 2 * p.bpass[i].ins_off,
                                   p.bpass[i].n_ins, true, true, p.Rb, 1, 1 << (p.k - p.Rb),
                                   p.lds_bwd, p.bpass[i].n_slots)});
  }
  return u;
}

namespace {

const char* const kJitOptions[] = {
    "--offload-arch=gfx950", "-O3", "-std=c++17",
    // no packed FP32 instructions in any device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    // keep the near-identical register cases apart (see build.py)
    "-mllvm", "-simplifycfg-sink-common=false", "-mllvm", "-simplifycfg-hoist-common=false"};

int compile_source(const std::string& src, std::vector<char>& code, std::string& log) {
  hiprtcProgram prog;
  if (hiprtcCreateProgram(&prog, src.c_str(), "vqc_jit.hip", kJitHeaderCount, kJitHeaderSources,
                          kJitHeaderNames) != HIPRTC_SUCCESS) {
    log = "hiprtcCreateProgram failed";
    return VQC_ERR_UNSUPPORTED;
  }
  const int nopt = (int)(sizeof(kJitOptions) / sizeof(kJitOptions[0]));
  const hiprtcResult rc = hiprtcCompileProgram(prog, nopt, kJitOptions);
  size_t n = 0;
  hiprtcGetProgramLogSize(prog, &n);
  log.assign(n, '\0');
  if (n) hiprtcGetProgramLog(prog, &log[0]);
  if (rc != HIPRTC_SUCCESS) {
    hiprtcDestroyProgram(&prog);
    return VQC_ERR_UNSUPPORTED;
  }
  size_t sz = 0;
  hiprtcGetCodeSize(prog, &sz);
  code.resize(sz);
  hiprtcGetCode(prog, code.data());
  hiprtcDestroyProgram(&prog);
  return VQC_OK;
}

// Compiles every source on a pool of host threads; returns the first failure.
int compile_all(const std::vector<const std::string*>& srcs, std::vector<std::vector<char>>& codes,
                std::string& log) {
  codes.assign(srcs.size(), {});
  std::vector<int> rcs(srcs.size(), VQC_OK);
  std::vector<std::string> logs(srcs.size());
  unsigned hw = std::thread::hardware_concurrency();
  const size_t nthreads = std::min<size_t>(srcs.size(), hw ? std::min(hw, 16u) : 4u);
  std::atomic<size_t> next{0};
  auto work = [&]() {
    for (size_t i; (i = next.fetch_add(1)) < srcs.size();)
      rcs[i] = compile_source(*srcs[i], codes[i], logs[i]);
  };
  std::vector<std::thread> pool;
  for (size_t t = 1; t < nthreads; ++t) pool.emplace_back(work);
  work();
  for (auto& th : pool) th.join();
  for (size_t i = 0; i < srcs.size(); ++i)
    if (rcs[i] != VQC_OK) {
      log = logs[i];
      return rcs[i];
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
  if (p.path == VQC_PATH_RESIDENT) {
    out.res_fwd = fns[0];
    out.res_bwd = fns[1];
  } else {
    out.pass_fwd.assign(fns.begin(), fns.begin() + p.fpass.size());
    out.pass_bwd.assign(fns.begin() + p.fpass.size(), fns.end());
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
