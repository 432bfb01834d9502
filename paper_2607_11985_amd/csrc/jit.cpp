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

// The training step: forward and adjoint sweeps in one kernel.
std::string step_unit(const Plan& p) {
  std::ostringstream o;
  o << "#include \"vqc_device.h\"\nnamespace vqc {\n";
  const int lanes = 1 << (p.k - p.R);
  const GradMode gm = grad_mode(lanes, p.P + p.F);
  emit_sched_struct(o, "SchedF", p, p.fwd.data(), (int)p.fwd.size() / 2, false, p.R, p.k, p.S, gm);
  emit_sched_struct(o, "SchedB", p, p.bwd.data(), (int)p.bwd.size() / 2, true, p.R, p.k, p.S, gm);
  o << "}  // namespace vqc\n"
    << "extern \"C\" __global__ void __launch_bounds__(" << p.WG << ") vqc_rs(const vqc::TileArgs A) {\n"
    << "  __shared__ __align__(16) unsigned char smem[" << lds_size(p.lds_step) << "];\n"
    << "  vqc::resident_step_body<" << p.WG << ", " << p.R
    << ", vqc::SchedF, vqc::SchedB>(A, smem);\n}\n";
  return o.str();
}

std::vector<JitUnit> jit_units(const Plan& p) {
  std::vector<JitUnit> u;
  if (p.path == VQC_PATH_RESIDENT) {
    u.push_back({"vqc_rf", kernel_unit(p, "vqc_rf", p.fwd.data(), (int)p.fwd.size() / 2, false,
                                       false, p.R, p.S, p.WG, p.lds_fwd, p.P + p.F)});
    u.push_back({"vqc_rb", kernel_unit(p, "vqc_rb", p.bwd.data(), (int)p.bwd.size() / 2, true,
                                       false, p.R, p.S, p.WG, p.lds_bwd, p.P + p.F)});
    u.push_back({"vqc_rs", step_unit(p)});
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
  if (p.path == VQC_PATH_RESIDENT) {
    out.res_fwd = fns[0];
    out.res_bwd = fns[1];
    out.res_step = fns[2];
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
