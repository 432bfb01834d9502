// api.cpp -- the C ABI declared in include/vqc.h.
#include <hip/hip_runtime_api.h>

#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "vqc.h"
#include "vqc_internal.h"

using vqc::Plan;

struct vqc_circuit {
  Plan plan;
  int device = -1;   // -1: host-only plan
  int engine = VQC_ENGINE_JIT;
  bool shared = false;  // one parameter vector for the batch
  vqc::JitKernels jit;
  void* blob = nullptr;
  size_t off_fwd = 0, off_bwd = 0, off_cols = 0, off_src = 0, off_idx = 0, off_cs = 0,
         off_maps = 0, off_pslots = 0, off_ma = 0, off_zm = 0, off_pc = 0;
  // Streaming path, generated kernels: the training step's own circuit, whose
  // plan leaves out the heads' rotations (Plan::product_head), or null.
  vqc_circuit* step = nullptr;
  ~vqc_circuit();
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

// Runs the caller's HIP work on the handle's device and restores the caller's
// current device afterwards.
class DeviceGuard {
 public:
  explicit DeviceGuard(int dev) {
    ok_ = hipGetDevice(&prev_) == hipSuccess;
    if (ok_ && prev_ != dev) ok_ = hipSetDevice(dev) == hipSuccess;
    else prev_ = -1;
  }
  ~DeviceGuard() {
    if (prev_ >= 0) (void)hipSetDevice(prev_);
  }
  bool ok() const { return ok_; }

 private:
  int prev_ = -1;
  bool ok_ = false;
};

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

template <typename T>
size_t append(std::vector<unsigned char>& blob, const std::vector<T>& v) {
  const size_t off = align_up(blob.size(), 256);
  blob.resize(off + std::max<size_t>(v.size() * sizeof(T), 1));
  if (!v.empty()) std::memcpy(blob.data() + off, v.data(), v.size() * sizeof(T));
  return off;
}

int64_t resident_blocks(const Plan& p, int64_t batch) { return (batch + p.S - 1) / p.S; }

size_t resident_state_bytes(const Plan& p, int64_t batch) {
  return (size_t)resident_blocks(p, batch) * (size_t)p.WG * ((size_t)1 << p.R) * 8;
}

// Streaming workspace: [E partials | tables | states ck[0..] | lambda x 2 |
// grad partials | cotangent].  Consecutive passes store the state in different
// memory layouts, so no pass writes the buffer it reads.  A training forward
// keeps every pass's output: pass i writes ck[i] (ck[nf - 1] is psi_G), and the
// adjoint's mirror of pass i reads it.  An inference forward alternates
// between ck[0] and ck[1].  The adjoint alternates lambda between l[0], l[1].
struct StreamLayout {
  size_t epart = 0, tabs = 0, gsig = 0, esig = 0;  // the table kernel's per-sample tables
  size_t ck0 = 0, state = 0;  // ck[i] = ck0 + i * state
  size_t end_inference = 0;
  size_t l[2] = {0, 0}, gpart = 0, end_training = 0;
  size_t cot = 0, end_step = 0;  // the training step's cotangent rows [B, n]
  size_t vpart = 0;              // product head: per-tile partials of v_q [B * 2^ng][NV]
  size_t ck(size_t i) const { return ck0 + i * state; }
};

// Head partials per tile (4 n floats rounded up to 16).
int head_nv(const Plan& p) { return (4 * p.n + 15) / 16 * 16; }

StreamLayout stream_layout(const Plan& p, int64_t batch) {
  StreamLayout L;
  const size_t tiles = (size_t)batch << p.ng;
  const size_t nocc = p.occ_src.size();
  const size_t nf = p.fpass.size();
  L.state = align_up((size_t)batch * ((size_t)1 << p.nq) * 8, 256);
  L.epart = 0;
  L.tabs = align_up(L.epart + tiles * (size_t)p.n * 4, 256);
  L.gsig = align_up(L.tabs + (size_t)batch * nocc * 8, 256);
  L.esig = align_up(L.gsig + (size_t)batch * nocc * 4, 256);
  L.ck0 = align_up(L.esig + (size_t)batch * p.n * 4, 256);
  L.end_inference = L.ck(std::min<size_t>(nf, 2));
  L.l[0] = L.ck(nf);
  L.l[1] = L.l[0] + L.state;
  L.gpart = L.l[1] + L.state;
  L.end_training = align_up(L.gpart + tiles * (size_t)(p.P + p.F) * 4, 256);
  L.cot = L.end_training;
  L.end_step = align_up(L.cot + (size_t)batch * (size_t)p.n * 4, 256);
  if (p.product_head) {
    L.vpart = L.end_step;
    L.end_step = align_up(L.vpart + tiles * (size_t)head_nv(p) * 4, 256);
  }
  return L;
}

// The end of the streaming layout of `batch` samples for `mode` (0 inference
// forward, 1 training forward (+ backward), 2 training step).
size_t stream_end(const Plan& p, int64_t batch, int mode) {
  const StreamLayout L = stream_layout(p, batch);
  return mode == 0 ? L.end_inference : mode == 1 ? L.end_training : L.end_step;
}

// The streaming calls run their batch as two halves, one on the caller's
// stream and one on a side stream, so that one half's passes fill the CUs the
// other's leave idle (the tail of each pass; in the training step also the
// HBM-bound forward of one half beside the VALU-bound adjoint of the other).
// Each half has a layout of its own: [half 0 | half 1].
bool split_batch(const Plan& p, int64_t batch) {
  return p.path == VQC_PATH_STREAM && batch >= 2;
}
int64_t first_half(int64_t batch) { return (batch + 1) / 2; }
size_t second_half_offset(const Plan& p, int64_t batch, int mode) {
  return align_up(stream_end(p, first_half(batch), mode), 256);
}

// mode: 0 inference forward, 1 training forward (+ backward), 2 training step
size_t required_bytes_core(const Plan& p, int64_t batch, int mode) {
  if (batch == 0) return 0;
  if (p.path == VQC_PATH_STREAM) {
    if (split_batch(p, batch))
      return second_half_offset(p, batch, mode) + stream_end(p, batch - first_half(batch), mode);
    return stream_end(p, batch, mode);
  }
  return mode == 1 ? resident_state_bytes(p, batch) : 0;
}

// With shared parameters the gradient passes through per-sample rows [B, P]
// placed after the rest of the workspace.
size_t shared_rows_offset(const Plan& p, int64_t batch, int mode) {
  return align_up(required_bytes_core(p, batch, mode), 256);
}

// Central differences (mode 3).  Slots are taken in chunks of fd_chunk (all
// of them on the resident path; on the streaming path as many as keep the
// shifted copies' states within 2 GiB).  Workspace: [streaming: the states and
// partials of one chunk's forward | the chunk's E rows [B * 2 chunk, n] |
// (shared parameters) the per-sample rows [B, P]].
constexpr size_t kFdStateBudget = size_t(2) << 30;

int fd_chunk(const Plan& p, int64_t batch) {
  const int NS = p.P + p.F;
  if (p.path == VQC_PATH_RESIDENT || NS == 0 || batch == 0) return NS;
  const size_t per_slot = (size_t)batch * 2 * 2 * ((size_t)1 << p.nq) * 8;  // two buffers
  const size_t c = kFdStateBudget / per_slot;
  return (int)std::max<size_t>(1, std::min<size_t>(c, (size_t)NS));
}

size_t fd_states_bytes(const Plan& p, int64_t batch) {
  if (p.path == VQC_PATH_RESIDENT) return 0;
  return stream_end(p, batch * 2 * fd_chunk(p, batch), 0);
}

size_t fd_rows_bytes(const Plan& p, int64_t batch) {
  return fd_states_bytes(p, batch) +
         align_up((size_t)batch * 2 * fd_chunk(p, batch) * p.n * 4, 256);
}

size_t required_bytes(const vqc_circuit* c, int64_t batch, int mode) {
  if (mode == 2 && c->step) c = c->step;  // the training step runs the step circuit
  const Plan& p = c->plan;
  if (batch == 0) return 0;
  if (mode == 3) return fd_rows_bytes(p, batch) + (c->shared ? (size_t)batch * p.P * 4 : 0);
  if (!c->shared || mode == 0 || p.P == 0) return required_bytes_core(p, batch, mode);
  return shared_rows_offset(p, batch, mode) + (size_t)batch * p.P * 4;
}

template <typename T>
const T* at(const vqc_circuit* c, size_t off) {
  return reinterpret_cast<const T*>(static_cast<const unsigned char*>(c->blob) + off);
}

vqc::TileArgs tile_args(const vqc_circuit* c, bool bwd, int64_t batch) {
  const Plan& p = c->plan;
  vqc::TileArgs a;
  std::memset(&a, 0, sizeof(a));
  a.ins = at<uint32_t>(c, bwd ? c->off_bwd : c->off_fwd);
  a.n_ins = (int32_t)((bwd ? p.bwd.size() : p.fwd.size()) / 2);
  a.cols = at<uint32_t>(c, c->off_cols);
  a.occ_src = at<int32_t>(c, c->off_src);
  a.occ_idx = at<int32_t>(c, c->off_idx);
  a.occ_cs = at<float>(c, c->off_cs);
  a.occ_ma = p.affine ? at<float>(c, c->off_ma) : nullptr;
  a.end_phys = at<uint8_t>(c, c->off_maps) + p.end_off;
  a.start_phys = at<uint8_t>(c, c->off_maps) + p.start_off;
  a.zmask = p.zmask.empty() ? nullptr : at<uint32_t>(c, c->off_zm);
  a.pcol = p.pcol.empty() ? nullptr : at<uint32_t>(c, c->off_pc);
  a.n_occ = (int32_t)p.occ_src.size();
  a.n_slots = p.P + p.F;
  a.P = p.P;
  a.F = p.F;
  a.pstride = c->shared ? 0 : p.P;
  a.n = p.n;
  a.k = p.k;
  a.t = p.t;
  a.S = p.S;
  a.G = p.G;
  a.B = batch;
  a.lds_tab = (uint32_t)p.lds_tab;
  a.lds_acc = (uint32_t)p.lds_acc;
  return a;
}

int check_runnable(const vqc_circuit* c) {
  if (!c) return fail(VQC_ERR_INVALID_ARG, "circuit handle is NULL");
  if (c->device < 0)
    return fail(VQC_ERR_INVALID_ARG, "circuit was compiled host-only (device = -1)");
  return VQC_OK;
}

int check_batch(const vqc_circuit* c, int64_t batch) {
  if (batch < 0) return fail(VQC_ERR_INVALID_ARG, "batch must be >= 0");
  const int64_t blocks = c->plan.path == VQC_PATH_STREAM ? (batch << c->plan.ng)
                                                         : resident_blocks(c->plan, batch);
  if (blocks > (int64_t)INT_MAX || batch > ((int64_t)1 << 40))
    return fail(VQC_ERR_TOO_LARGE, "batch too large for one launch");
  return VQC_OK;
}

vqc::PassArgs pass_args(const vqc_circuit* c, const vqc::PassPlan& pp, bool bwd, int64_t batch) {
  const Plan& p = c->plan;
  vqc::PassArgs a;
  std::memset(&a, 0, sizeof(a));
  a.ins = at<uint32_t>(c, bwd ? c->off_bwd : c->off_fwd) + 2 * (size_t)pp.ins_off;
  a.n_ins = pp.n_ins;
  a.cols = at<uint32_t>(c, c->off_cols);
  a.io = a.cols + pp.io_off;
  a.io_out = a.cols + pp.io_out_off;
  a.io_lin = a.cols + pp.io_lin_off;
  a.io_lout = a.cols + pp.io_lout_off;
  a.start_phys = at<uint8_t>(c, c->off_maps) + pp.start_off;
  a.end_phys = at<uint8_t>(c, c->off_maps) + pp.end_off;
  a.zmask = p.zmask.empty() ? nullptr : at<uint32_t>(c, c->off_zm);
  a.pslots = at<int32_t>(c, c->off_pslots) + pp.slots_off;
  a.n_pslots = pp.n_slots;
  a.flags = pp.flags;
  a.occ_src = at<int32_t>(c, c->off_src);
  a.occ_idx = at<int32_t>(c, c->off_idx);
  a.occ_cs = at<float>(c, c->off_cs);
  a.occ_ma = p.affine ? at<float>(c, c->off_ma) : nullptr;
  a.n_occ = (int32_t)p.occ_src.size();
  a.n_slots = p.P + p.F;
  a.P = p.P;
  a.F = p.F;
  a.pstride = c->shared ? 0 : p.P;
  a.n = p.n;
  a.k = p.k;
  a.ng = p.ng;
  a.B = batch;
  a.lds_tab = (uint32_t)p.lds_tab;
  a.lds_acc = (uint32_t)p.lds_acc;
  return a;
}

int hip_fail(const char* what, int rc) {
  return fail(VQC_ERR_HIP, std::string(what) + " failed: " + hipGetErrorString((hipError_t)rc));
}

int check_rows(const vqc_circuit* c, const float* params, const float* inputs) {
  if (c->plan.P > 0 && !params) return fail(VQC_ERR_INVALID_ARG, "params is NULL but P > 0");
  if (c->plan.F > 0 && !inputs) return fail(VQC_ERR_INVALID_ARG, "inputs is NULL but F > 0");
  return VQC_OK;
}

int check_workspace(const void* workspace, size_t bytes, size_t need, const char* what) {
  if (need == 0) return VQC_OK;
  if (!workspace || bytes < need) return fail(VQC_ERR_WORKSPACE, what);
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(VQC_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return VQC_OK;
}

// The generated kernels' per-sample tables, once per call before the passes
// (the passes read them through PassArgs::tabs / gsig / esig).
int launch_tables(const vqc_circuit* c, vqc::PassArgs a, int64_t batch, void* stream) {
  if (!c->jit.tables || batch == 0) return 0;
  return vqc::jit_launch(c->jit.tables, batch, vqc::kTableThreads, &a, sizeof(a), stream);
}

void set_tables(vqc::PassArgs& a, unsigned char* ws, const StreamLayout& L) {
  a.tabs = reinterpret_cast<float*>(ws + L.tabs);
  a.gsig = reinterpret_cast<float*>(ws + L.gsig);
  a.esig = reinterpret_cast<float*>(ws + L.esig);
}

// The library's side stream on `device` (the caller makes it current),
// created on first use with the default priority and kept until exit.
int side_stream(int device, hipStream_t* out) {
  static std::mutex mu;
  static hipStream_t streams[vqc::kScratchDevices] = {};
  *out = nullptr;
  if (device < 0 || device >= vqc::kScratchDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!streams[device]) {
    hipStream_t s = nullptr;
    const hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    if (e != hipSuccess) return (int)e;
    streams[device] = s;
  }
  *out = streams[device];
  return 0;
}

template <typename T>
T* rows_at(T* base, int64_t row, int64_t width) {
  return base ? base + row * width : nullptr;
}

// Runs f(first row, rows, half's workspace offset index, stream) for the two
// halves of a streaming call: the first on `stream`, the second on the side
// stream, which waits for the work queued on `stream` before the call;
// `stream` then waits for the second half, so work queued on it later sees
// the whole call.
template <typename F>
int on_two_streams(const vqc_circuit* c, int64_t batch, void* stream, F&& f) {
  const int64_t b0 = first_half(batch), b1 = batch - b0;
  hipStream_t side = nullptr;
  int rc = side_stream(c->device, &side);
  if (rc) return hip_fail("side stream creation", rc);
  hipEvent_t fork = nullptr, join = nullptr;
  if ((rc = hipEventCreateWithFlags(&fork, hipEventDisableTiming)))
    return hip_fail("event creation", rc);
  if ((rc = hipEventCreateWithFlags(&join, hipEventDisableTiming))) {
    (void)hipEventDestroy(fork);
    return hip_fail("event creation", rc);
  }
  struct Events {
    hipEvent_t a, b;
    ~Events() {
      (void)hipEventDestroy(a);  // released once the device has passed them
      (void)hipEventDestroy(b);
    }
  } events{fork, join};
  if ((rc = hipEventRecord(fork, (hipStream_t)stream)) ||
      (rc = hipStreamWaitEvent(side, fork, 0)))
    return hip_fail("stream fork", rc);
  rc = f((int64_t)0, b0, 0, stream);
  if (rc) return rc;
  const int rc1 = f(b0, b1, 1, (void*)side);
  // join even after a failed launch, so that `stream` never runs ahead of
  // what the side stream already holds
  if ((rc = hipEventRecord(join, side)) || (rc = hipStreamWaitEvent((hipStream_t)stream, join, 0)))
    return hip_fail("stream join", rc);
  return rc1;
}

// The training step's additions to its forward: the loss head (its cotangent
// rows computed with the <Z> reduction) and the adjoint's gradient partials,
// cleared by the table kernel.
struct StepHead {
  int32_t kind;
  int64_t norm;
  const float* target;
  float* cot;
};

// Streaming forward: every pass (the first starts from |0...0> or reads psi0),
// then the <Z> reduction into expvals; the last pass writes probs.  fd_slots > 0:
// the batch is the central differences' shifted copies of slots fd_base ..
int stream_forward(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                   float* expvals, unsigned char* ws, void* stream, bool keep,
                   const void* psi0 = nullptr, float* probs = nullptr, int fd_base = 0,
                   int fd_slots = 0, float fd_h = 0.f, const StepHead* step = nullptr) {
  const Plan& p = c->plan;
  const StreamLayout L = stream_layout(p, batch);
  int rc = 0;
  for (const vqc::PassPlan& pp : p.fpass) {
    vqc::PassArgs a = pass_args(c, pp, false, batch);
    const size_t i = &pp - p.fpass.data();
    a.params = params;
    a.inputs = inputs;
    set_tables(a, ws, L);
    a.psi_src = ws + (keep ? L.ck(i ? i - 1 : 0) : L.ck((i + 1) % 2));
    a.psi_dst = ws + (keep ? L.ck(i) : L.ck(i % 2));
    if (psi0 && (a.flags & vqc::PF_INIT)) {
      if (p.product_head) return fail(VQC_ERR_UNSUPPORTED, "internal: Psi_0 with a product head");
      a.flags &= ~vqc::PF_INIT;
      a.psi_src = psi0;
      a.psi0_in = 1;
    }
    if (a.flags & vqc::PF_ZPART) a.probs = probs;
    a.fd_base = fd_base;
    a.fd_slots = fd_slots;
    a.fd_h = fd_h;
    a.epart = reinterpret_cast<float*>(ws + L.epart);
    if (i == 0) {
      vqc::PassArgs t = a;
      if (step) t.gpart = reinterpret_cast<float*>(ws + L.gpart);
      rc = launch_tables(c, t, batch, stream);
      if (rc) return hip_fail("table kernel launch", rc);
    }
    rc = c->engine == VQC_ENGINE_JIT
             ? vqc::jit_launch(c->jit.pass_fwd[i], batch << p.ng, 1 << (p.k - p.Rf), &a, sizeof(a),
                               stream)
             : vqc::launch_stream_pass(p, false, a, batch << p.ng, stream);
    if (rc) return hip_fail("forward pass launch", rc);
  }
  if (!expvals) return VQC_OK;
  const float* epart = reinterpret_cast<const float*>(ws + L.epart);
  rc = step ? vqc::launch_reduce_e_loss(batch, p.ng, p.n, epart, expvals, step->kind, step->norm,
                                        step->target, step->cot, stream)
            : vqc::launch_reduce_e(batch, p.ng, p.n, epart, expvals, stream);
  if (rc) return hip_fail("expectation reduction launch", rc);
  return VQC_OK;
}

// Streaming adjoint: clear the partials (the table kernel does, when there is
// one), every pass (the first reads the saved psi_G and leaves it intact), then
// the reduction into dparams / dinputs (with a product head: the head
// kernel's).  prepared: the training step's forward wrote this call's tables
// and cleared the partials.
int stream_backward(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                    const float* grad_out, unsigned char* ws, float* dp, float* dx, void* stream,
                    bool prepared = false) {
  const Plan& p = c->plan;
  const StreamLayout L = stream_layout(p, batch);
  float* gpart = reinterpret_cast<float*>(ws + L.gpart);
  int rc = 0;
  if (!prepared && !c->jit.tables &&
      (rc = vqc::launch_fill_zero(gpart, (batch << p.ng) * (int64_t)(p.P + p.F), stream)))
    return hip_fail("gradient partial clear", rc);
  bool first = !prepared;
  for (const vqc::PassPlan& pp : p.bpass) {
    vqc::PassArgs a = pass_args(c, pp, true, batch);
    const size_t j = &pp - p.bpass.data();
    a.params = params;
    a.inputs = inputs;
    a.grad_out = grad_out;
    a.psi_src = ws + L.ck(p.fpass.size() - 1 - j);  // the state its forward pass saved
    a.psi_dst = nullptr;
    a.lam_src = ws + L.l[(j + 1) % 2];
    a.lam_dst = ws + L.l[j % 2];
    a.gpart = gpart;
    a.vpart = p.product_head ? reinterpret_cast<float*>(ws + L.vpart) : nullptr;
    set_tables(a, ws, L);
    if (first) {
      rc = launch_tables(c, a, batch, stream);
      if (rc) return hip_fail("table kernel launch", rc);
    }
    rc = c->engine == VQC_ENGINE_JIT
             ? vqc::jit_launch(c->jit.pass_bwd[j], batch << p.ng, 1 << (p.k - p.Rb), &a, sizeof(a),
                               stream)
             : vqc::launch_stream_pass(p, true, a, batch << p.ng, stream);
    if (rc) return hip_fail("backward pass launch", rc);
    first = false;
  }
  if (p.product_head) {
    // the heads' gradients, and every slot's sum over the tiles, into the rows
    vqc::PassArgs a = pass_args(c, p.bpass.back(), true, batch);
    a.gpart = gpart;
    a.vpart = reinterpret_cast<float*>(ws + L.vpart);
    a.dparams = dp;
    a.dinputs = dx;
    set_tables(a, ws, L);
    rc = c->jit.head_finish ? vqc::jit_launch(c->jit.head_finish, batch, vqc::kHeadThreads, &a,
                                              sizeof(a), stream)
                            : (int)hipErrorInvalidDeviceFunction;
    return rc ? hip_fail("head gradient launch", rc) : VQC_OK;
  }
  rc = vqc::launch_reduce_grad(batch, p.ng, p.P + p.F, p.P, p.F, gpart, dp, dx, stream);
  if (rc) return hip_fail("gradient reduction launch", rc);
  return VQC_OK;
}

}  // namespace

vqc_circuit::~vqc_circuit() {
  delete step;
  if (blob) {
    DeviceGuard g(device);
    (void)hipFree(blob);
  }
}

namespace {

// The plan's tables in device memory (one allocation) and its kernels: the
// generated ones, or the fixed ones' attributes.
int load_device(vqc_circuit* c, std::string& msg) {
  const Plan& p = c->plan;
  std::vector<unsigned char> blob;
  c->off_fwd = append(blob, p.fwd);
  c->off_bwd = append(blob, p.bwd);
  c->off_cols = append(blob, p.cols);
  c->off_src = append(blob, p.occ_src);
  c->off_idx = append(blob, p.occ_idx);
  c->off_cs = append(blob, p.occ_cs);
  c->off_ma = append(blob, p.occ_ma);
  c->off_maps = append(blob, p.maps);
  c->off_pslots = append(blob, p.pslots);
  c->off_zm = append(blob, p.zmask);
  c->off_pc = append(blob, p.pcol);
  DeviceGuard g(c->device);
  if (!g.ok()) {
    msg = "hipSetDevice failed";
    return VQC_ERR_HIP;
  }
  if (hipMalloc(&c->blob, blob.size()) != hipSuccess) {
    c->blob = nullptr;
    msg = "hipMalloc of the schedule failed";
    return VQC_ERR_HIP;
  }
  if (hipMemcpy(c->blob, blob.data(), blob.size(), hipMemcpyHostToDevice) != hipSuccess) {
    msg = "copy of the schedule failed";
    return VQC_ERR_HIP;
  }
  if (c->engine == VQC_ENGINE_JIT) return vqc::jit_build(p, c->device, c->jit, msg);
  const int rc = vqc::prepare_kernels(p);
  if (rc != 0) {
    msg = std::string("hipFuncSetAttribute failed: ") + hipGetErrorString((hipError_t)rc);
    return VQC_ERR_HIP;
  }
  return VQC_OK;
}

}  // namespace

extern "C" {

const char* vqc_last_error(void) { return g_err.c_str(); }

int vqc_compile(const vqc_op* ops, int32_t n_ops, int32_t n_qubits, int32_t n_params,
                int32_t n_inputs, const vqc_compile_opts* opts, vqc_circuit** out) {
  if (!out) return fail(VQC_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (n_ops < 0) return fail(VQC_ERR_INVALID_ARG, "n_ops must be >= 0");
  if (n_ops > 0 && !ops) return fail(VQC_ERR_INVALID_ARG, "ops is NULL");
  if (n_ops > (1 << 20)) return fail(VQC_ERR_TOO_LARGE, "more than 2^20 gates");
  int device = 0, path = VQC_PATH_AUTO, reg_bits = 0, engine = VQC_ENGINE_JIT, tile = 0;
  bool shared = false;
  if (opts) {
    for (int r : opts->reserved)
      if (r != 0) return fail(VQC_ERR_INVALID_ARG, "reserved option fields must be zero");
    device = opts->device;
    path = opts->path;
    reg_bits = opts->reg_bits;
    engine = opts->engine;
    if (engine != VQC_ENGINE_JIT && engine != VQC_ENGINE_INTERP)
      return fail(VQC_ERR_INVALID_ARG, "unknown engine option");
    if (opts->shared_params != 0 && opts->shared_params != 1)
      return fail(VQC_ERR_INVALID_ARG, "shared_params must be 0 or 1");
    shared = opts->shared_params == 1;
    tile = opts->tile_qubits;
    if (tile != 0 && tile != 12 && tile != 13 && tile != 14)
      return fail(VQC_ERR_INVALID_ARG, "tile_qubits must be 0 (default), 12, 13 or 14");
    if ((tile == 12 || tile == 13) && engine != VQC_ENGINE_JIT)
      return fail(VQC_ERR_UNSUPPORTED, "12- and 13-qubit tiles need the generated kernels");
    if (path < VQC_PATH_AUTO || path > VQC_PATH_STREAM)
      return fail(VQC_ERR_INVALID_ARG, "unknown path option");
  } else if (hipGetDevice(&device) != hipSuccess) {
    return fail(VQC_ERR_HIP, "hipGetDevice failed");
  }
  std::vector<vqc::HostOp> hops((size_t)n_ops);
  for (int k = 0; k < n_ops; ++k) {
    const vqc_op& o = ops[k];
    vqc::HostOp& h = hops[k];
    h.kind = o.kind;
    for (int s = 0; s < 3; ++s) {
      h.w[s] = o.wires[s];
      h.src[s] = o.src[s];
      h.idx[s] = o.idx[s];
      h.val[s] = o.val[s];
      h.mul[s] = o.mul[s];
    }
  }
  vqc_circuit* c = new (std::nothrow) vqc_circuit();
  if (!c) return fail(VQC_ERR_OOM, "out of host memory");
  std::string msg;
  int rc = vqc::build_plan(hops, n_qubits, n_params, n_inputs, path, reg_bits, c->plan, msg,
                           engine == VQC_ENGINE_JIT, tile);
  if (rc != 0) {
    delete c;
    return fail(rc, msg);
  }
  // Default tiles of the generated kernels: 12 qubits unless that takes more
  // than a quarter more passes than 13.  Four workgroups per CU instead of two
  // hide more latency: measured 1.6-4 % faster on the 14-qubit re-uploading
  // workload (same passes) and 3.5 % on the 16-qubit ring (29 passes, not 24).
  if (engine == VQC_ENGINE_JIT && tile == 0 && c->plan.path == VQC_PATH_STREAM) {
    Plan p12;
    std::string msg12;
    const size_t n13 = c->plan.fpass.size() + c->plan.bpass.size();
    if (vqc::build_plan(hops, n_qubits, n_params, n_inputs, path, reg_bits, p12, msg12, true, 12) ==
            0 &&
        4 * (p12.fpass.size() + p12.bpass.size()) <= 5 * n13)
      c->plan = std::move(p12);
  }
  // The generated adjoint passes hold 16 amplitudes per thread (the batched
  // gradient reduction fits there); reg_bits = 5 asks for 32.  32 halve the
  // workgroups per CU that hide each pass's loads and stores.  Measured on one
  // box: the 14-qubit re-uploading workload 11.58 ms per step at 32 (26
  // exchanges) against 11.10 ms at 16 (33 exchanges); the 16-qubit ring was
  // 13-25 % slower at 32.
  c->device = device;
  c->engine = engine;
  c->shared = shared;
  // The streaming training step builds the product state after every qubit's
  // head instead of running the heads' rotations (generated kernels; the
  // heads' exact angles come from the table kernel).  Measured on the 16-qubit
  // ring and the 14-qubit re-uploading workloads: without their heads' gates
  // the steps take 11.5 % and 9.5 % less time.
  if (engine == VQC_ENGINE_JIT && c->plan.path == VQC_PATH_STREAM) {
    Plan sp;
    std::string msg_s;
    if (vqc::build_step_plan(c->plan, sp, msg_s) == 0 && vqc::stream_tables_fit(sp)) {
      c->step = new (std::nothrow) vqc_circuit();
      if (!c->step) {
        delete c;
        return fail(VQC_ERR_OOM, "out of host memory");
      }
      c->step->plan = std::move(sp);
      c->step->device = device;
      c->step->engine = engine;
      c->step->shared = shared;
    }
  }
  if (device >= 0) {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device >= count) {
      delete c;
      return fail(VQC_ERR_INVALID_ARG, "no HIP device " + std::to_string(device));
    }
    rc = load_device(c, msg);
    if (rc == VQC_OK && c->step) rc = load_device(c->step, msg);
    if (rc != VQC_OK) {
      delete c;
      return fail(rc, msg);
    }
  }
  *out = c;
  return VQC_OK;
}

int vqc_parse_qasm(const char* source, const char* input_names, vqc_op* ops, int32_t capacity,
                   int32_t* n_ops, int32_t* n_qubits, int32_t* n_params, int32_t* n_inputs) {
  if (!n_ops || !n_qubits || !n_params || !n_inputs)
    return fail(VQC_ERR_INVALID_ARG, "an output count pointer is NULL");
  if (capacity < 0 || (capacity > 0 && !ops))
    return fail(VQC_ERR_INVALID_ARG, "ops is NULL or capacity is negative");
  std::vector<vqc_op> v;
  int nq = 0, np = 0, ni = 0;
  std::string msg;
  const int rc = vqc::parse_qasm(source, input_names, v, nq, np, ni, msg);
  if (rc) return fail(rc, msg);
  *n_ops = (int32_t)v.size();
  *n_qubits = nq;
  *n_params = np;
  *n_inputs = ni;
  if (ops && (int64_t)v.size() > capacity)
    return fail(VQC_ERR_TOO_LARGE, "ops capacity " + std::to_string(capacity) + " < " +
                                       std::to_string(v.size()) + " gates");
  if (ops && !v.empty()) std::memcpy(ops, v.data(), v.size() * sizeof(vqc_op));
  return VQC_OK;
}

int vqc_compile_qasm(const char* source, const char* input_names, const vqc_compile_opts* opts,
                     vqc_circuit** out) {
  if (!out) return fail(VQC_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  std::vector<vqc_op> v;
  int nq = 0, np = 0, ni = 0;
  std::string msg;
  const int rc = vqc::parse_qasm(source, input_names, v, nq, np, ni, msg);
  if (rc) return fail(rc, msg);
  return vqc_compile(v.data(), (int32_t)v.size(), nq, np, ni, opts, out);
}

void vqc_destroy(vqc_circuit* c) { delete c; }

size_t vqc_workspace_bytes(const vqc_circuit* c, int64_t batch, int32_t training) {
  if (!c || batch < 0 || training < 0 || training > 3) return (size_t)-1;
  return required_bytes(c, batch, training);
}

int vqc_forward(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                float* expvals, void* workspace, size_t workspace_bytes, void* stream) {
  if (c && batch > 0 && !expvals) return fail(VQC_ERR_INVALID_ARG, "expvals is NULL");
  return vqc_forward_ex(c, batch, params, inputs, nullptr, expvals, nullptr, workspace,
                        workspace_bytes, stream);
}

int vqc_forward_ex(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                   const void* psi0, float* expvals, float* probs, void* workspace,
                   size_t workspace_bytes, void* stream) {
  int rc = check_runnable(c);
  if (rc) return rc;
  if ((rc = check_batch(c, batch))) return rc;
  if (batch == 0) return VQC_OK;
  if ((rc = check_rows(c, params, inputs))) return rc;
  if (!expvals && !probs) return fail(VQC_ERR_INVALID_ARG, "expvals and probs are both NULL");
  if (psi0 && reinterpret_cast<uintptr_t>(psi0) % 8)
    return fail(VQC_ERR_INVALID_ARG, "psi0 must be 8-byte aligned (complex64)");
  if (probs && reinterpret_cast<uintptr_t>(probs) % 4)
    return fail(VQC_ERR_INVALID_ARG, "probs must be 4-byte aligned");
  const Plan& p = c->plan;
  if (p.path == VQC_PATH_STREAM && !workspace)
    return fail(VQC_ERR_WORKSPACE, "the streaming path needs a workspace (states live in HBM)");
  if (workspace) {
    const int mode = p.path == VQC_PATH_RESIDENT ? 1 : 0;
    if ((rc = check_workspace(workspace, workspace_bytes, required_bytes(c, batch, mode),
                              mode ? "workspace smaller than vqc_workspace_bytes(c, batch, 1)"
                                   : "workspace smaller than vqc_workspace_bytes(c, batch, 0)")))
      return rc;
  }
  DeviceGuard g(c->device);
  if (!g.ok()) return fail(VQC_ERR_HIP, "hipSetDevice failed");
  if (p.path == VQC_PATH_STREAM) {
    // a workspace that holds the training layout keeps every pass's state
    const bool keep = workspace_bytes >= required_bytes_core(p, batch, 1);
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    if (!split_batch(p, batch))
      return stream_forward(c, batch, params, inputs, expvals, ws, stream, keep, psi0, probs);
    const int64_t P = c->shared ? 0 : p.P, N = (int64_t)1 << p.n;
    const size_t off = second_half_offset(p, batch, keep ? 1 : 0);
    return on_two_streams(c, batch, stream, [&](int64_t b0, int64_t nb, int h, void* st) {
      const void* s0 = psi0 ? static_cast<const unsigned char*>(psi0) + b0 * N * 8 : nullptr;
      return stream_forward(c, nb, rows_at(params, b0, P), rows_at(inputs, b0, p.F),
                            rows_at(expvals, b0, p.n), ws + h * off, st, keep, s0,
                            rows_at(probs, b0, N));
    });
  }
  vqc::TileArgs a = tile_args(c, false, batch);
  a.params = params;
  a.inputs = inputs;
  a.expvals = expvals;
  a.ws = workspace;
  a.psi0 = psi0;
  a.probs = probs;
  rc = c->engine == VQC_ENGINE_JIT
           ? vqc::jit_launch(c->jit.res_fwd, resident_blocks(p, batch), p.WG, &a, sizeof(a), stream)
           : vqc::launch_resident_forward(p, a, resident_blocks(p, batch), stream);
  if (rc) return hip_fail("forward launch", rc);
  return VQC_OK;
}

int vqc_backward(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                 const float* grad_out, void* workspace, size_t workspace_bytes, float* dparams,
                 float* dinputs, void* stream) {
  int rc = check_runnable(c);
  if (rc) return rc;
  if ((rc = check_batch(c, batch))) return rc;
  if (batch == 0) return VQC_OK;
  if ((rc = check_rows(c, params, inputs))) return rc;
  if (!grad_out) return fail(VQC_ERR_INVALID_ARG, "grad_out is NULL");
  const Plan& p = c->plan;
  if ((rc = check_workspace(workspace, workspace_bytes, required_bytes(c, batch, 1),
                            "backward needs the workspace of a training forward")))
    return rc;
  DeviceGuard g(c->device);
  if (!g.ok()) return fail(VQC_ERR_HIP, "hipSetDevice failed");
  float* dp = p.P > 0 ? dparams : nullptr;
  float* dx = p.F > 0 ? dinputs : nullptr;
  // shared parameters: per-sample rows first, summed over the batch after
  float* rows = (c->shared && dp) ? reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) +
                                                             shared_rows_offset(p, batch, 1))
                                  : nullptr;
  if (p.path == VQC_PATH_STREAM) {
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    float* dprows = rows ? rows : dp;
    if (split_batch(p, batch)) {
      const int64_t P = c->shared ? 0 : p.P;
      const size_t off = second_half_offset(p, batch, 1);
      rc = on_two_streams(c, batch, stream, [&](int64_t b0, int64_t nb, int h, void* st) {
        return stream_backward(c, nb, rows_at(params, b0, P), rows_at(inputs, b0, p.F),
                               rows_at(grad_out, b0, p.n), ws + h * off,
                               rows_at(dprows, b0, p.P), rows_at(dx, b0, p.F), st);
      });
    } else {
      rc = stream_backward(c, batch, params, inputs, grad_out, ws, dprows, dx, stream);
    }
    if (rc || !rows) return rc;
    rc = vqc::launch_sum_rows(batch, p.P, rows, dp, stream);
    return rc ? hip_fail("parameter gradient sum", rc) : VQC_OK;
  }
  vqc::TileArgs a = tile_args(c, true, batch);
  a.params = params;
  a.inputs = inputs;
  a.ws = workspace;
  a.grad_out = grad_out;
  a.dparams = rows ? rows : dp;
  a.dinputs = dx;
  rc = c->engine == VQC_ENGINE_JIT
           ? vqc::jit_launch(c->jit.res_bwd, resident_blocks(p, batch), p.WG, &a, sizeof(a), stream)
           : vqc::launch_resident_backward(p, a, resident_blocks(p, batch), stream);
  if (rc) return hip_fail("backward launch", rc);
  if (rows && (rc = vqc::launch_sum_rows(batch, p.P, rows, dp, stream)))
    return hip_fail("parameter gradient sum", rc);
  return VQC_OK;
}

}  // extern "C"

namespace {

// The argument checks of vqc_train_step (those that need no workspace).
int check_step_args(const vqc_circuit* c, int64_t batch, const float* params,
                    const float* inputs, int32_t loss_kind, const float* target,
                    const float* expvals) {
  int rc = check_runnable(c);
  if (rc) return rc;
  if (loss_kind < VQC_LOSS_SUM || loss_kind > VQC_LOSS_MSE_MEANZ)
    return fail(VQC_ERR_INVALID_ARG, "unknown loss kind");
  if ((rc = check_batch(c, batch))) return rc;
  if (batch == 0) return VQC_OK;
  if ((rc = check_rows(c, params, inputs))) return rc;
  if (!expvals) return fail(VQC_ERR_INVALID_ARG, "expvals is NULL");
  if ((loss_kind == VQC_LOSS_MSE_Z0 || loss_kind == VQC_LOSS_MSE_MEANZ) && !target)
    return fail(VQC_ERR_INVALID_ARG, "MSE losses need a target");
  return VQC_OK;
}

// Streaming forward, loss cotangent and adjoint of `batch` rows of a batch of
// `norm` samples (pointers at the rows' start, the workspace laid out for
// `batch`).
int stream_step(const vqc_circuit* c, int64_t batch, int64_t norm, const float* params,
                const float* inputs, int32_t loss_kind, const float* target, float* expvals,
                float* grad_out, float* dp, float* dx, unsigned char* ws, void* stream) {
  const Plan& p = c->plan;
  float* cot = grad_out ? grad_out : reinterpret_cast<float*>(ws + stream_layout(p, batch).cot);
  const StepHead sh{loss_kind, norm, target, cot};
  int rc = stream_forward(c, batch, params, inputs, expvals, ws, stream, true, nullptr, nullptr, 0,
                          0, 0.f, &sh);
  if (rc) return rc;
  // with a table kernel the forward's tables serve the adjoint, and it cleared the partials
  return stream_backward(c, batch, params, inputs, cot, ws, dp, dx, stream,
                         c->jit.tables != nullptr);
}

// The training step on a checked, large enough workspace, with the handle's
// device current.  split: the streaming path may run the two halves of the
// batch on two streams (the workspace then holds the split layout).
int train_step_impl(const vqc_circuit* c, int64_t batch, const float* params,
                    const float* inputs, int32_t loss_kind, const float* target, float* expvals,
                    float* grad_out, float* dparams, float* dinputs, void* workspace,
                    void* stream, bool split) {
  const Plan& p = c->plan;
  // with a product head the streaming step runs the circuit planned without the heads
  const vqc_circuit* sc = c->step ? c->step : c;
  int rc = 0;
  float* dp = p.P > 0 ? dparams : nullptr;
  float* dx = p.F > 0 ? dinputs : nullptr;
  float* rows = (c->shared && dp) ? reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) +
                                                             shared_rows_offset(sc->plan, batch, 2))
                                  : nullptr;
  if (p.path == VQC_PATH_STREAM) {
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    float* dprows = rows ? rows : dp;
    if (split && split_batch(p, batch)) {
      const int64_t P = c->shared ? 0 : p.P;
      const size_t off = second_half_offset(sc->plan, batch, 2);
      rc = on_two_streams(c, batch, stream, [&](int64_t b0, int64_t nb, int h, void* st) {
        return stream_step(sc, nb, batch, rows_at(params, b0, P), rows_at(inputs, b0, p.F),
                           loss_kind, rows_at(target, b0, 1), rows_at(expvals, b0, p.n),
                           rows_at(grad_out, b0, p.n), rows_at(dprows, b0, p.P),
                           rows_at(dx, b0, p.F), ws + h * off, st);
      });
    } else {
      rc = stream_step(sc, batch, batch, params, inputs, loss_kind, target, expvals, grad_out,
                       dprows, dx, ws, stream);
    }
    if (rc || !rows) return rc;
    rc = vqc::launch_sum_rows(batch, p.P, rows, dp, stream);
    return rc ? hip_fail("parameter gradient sum", rc) : VQC_OK;
  }
  vqc::TileArgs a = tile_args(c, false, batch);
  a.ins_b = at<uint32_t>(c, c->off_bwd);
  a.n_ins_b = (int32_t)(p.bwd.size() / 2);
  a.params = params;
  a.inputs = inputs;
  a.expvals = expvals;
  a.loss = loss_kind;
  a.target = target;
  a.cot_out = grad_out;
  a.dparams = rows ? rows : dp;
  a.dinputs = dx;
  a.lds_e = (uint32_t)p.lds_e;
  rc = c->engine == VQC_ENGINE_JIT
           ? vqc::jit_launch(c->jit.res_step, resident_blocks(p, batch), p.WG, &a, sizeof(a),
                             stream)
           : vqc::launch_resident_step(p, a, resident_blocks(p, batch), stream);
  if (rc) return hip_fail("training step launch", rc);
  if (rows && (rc = vqc::launch_sum_rows(batch, p.P, rows, dp, stream)))
    return hip_fail("parameter gradient sum", rc);
  return VQC_OK;
}

}  // namespace

extern "C" {

int vqc_train_step(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                   int32_t loss_kind, const float* target, float* expvals, float* grad_out,
                   float* dparams, float* dinputs, void* workspace, size_t workspace_bytes,
                   void* stream) {
  int rc = check_step_args(c, batch, params, inputs, loss_kind, target, expvals);
  if (rc || batch == 0) return rc;
  if ((rc = check_workspace(workspace, workspace_bytes, required_bytes(c, batch, 2),
                            "workspace smaller than vqc_workspace_bytes(c, batch, 2)")))
    return rc;
  DeviceGuard g(c->device);
  if (!g.ok()) return fail(VQC_ERR_HIP, "hipSetDevice failed");
  return train_step_impl(c, batch, params, inputs, loss_kind, target, expvals, grad_out, dparams,
                         dinputs, workspace, stream, true);
}

int vqc_train_step_noalloc(const vqc_circuit* c, int64_t batch, const float* params,
                           const float* inputs, int32_t loss_kind, const float* target,
                           float* expvals, float* grad_out, float* dparams, float* dinputs,
                           void* stream) {
  int rc = check_step_args(c, batch, params, inputs, loss_kind, target, expvals);
  if (rc || batch == 0) return rc;
  const size_t need = required_bytes(c, batch, 2);
  if (need > (size_t)VQC_NOALLOC_SCRATCH_BYTES)
    return fail(VQC_ERR_TOO_LARGE,
                "the step needs " + std::to_string(need) + " bytes of workspace; the static "
                "scratch of vqc_train_step_noalloc holds " +
                    std::to_string((size_t)VQC_NOALLOC_SCRATCH_BYTES));
  DeviceGuard g(c->device);
  if (!g.ok()) return fail(VQC_ERR_HIP, "hipSetDevice failed");
  void* ws = nullptr;
  if (need > 0 && (rc = vqc::scratch_pointer(c->device, &ws)))
    return hip_fail("lookup of the static scratch", rc);
  // one stream: the side stream and its events would be created on first use
  return train_step_impl(c, batch, params, inputs, loss_kind, target, expvals, grad_out, dparams,
                         dinputs, ws, stream, false);
}

int vqc_fd_backward(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                    const float* grad_out, float h, void* workspace, size_t workspace_bytes,
                    float* dparams, float* dinputs, void* stream) {
  int rc = check_runnable(c);
  if (rc) return rc;
  const Plan& p = c->plan;
  if (!(h > 0.f) || !std::isfinite(h)) return fail(VQC_ERR_INVALID_ARG, "h must be finite and > 0");
  if ((rc = check_batch(c, batch))) return rc;
  const int NS = p.P + p.F;
  if (batch == 0 || NS == 0) return VQC_OK;
  if ((rc = check_rows(c, params, inputs))) return rc;
  if (!grad_out) return fail(VQC_ERR_INVALID_ARG, "grad_out is NULL");
  const int chunk = fd_chunk(p, batch);
  const int64_t virt = batch * 2 * chunk;
  if ((rc = check_batch(c, virt))) return rc;
  if ((rc = check_workspace(workspace, workspace_bytes, required_bytes(c, batch, 3),
                            "workspace smaller than vqc_workspace_bytes(c, batch, 3)")))
    return rc;
  DeviceGuard g(c->device);
  if (!g.ok()) return fail(VQC_ERR_HIP, "hipSetDevice failed");
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  float* ev = reinterpret_cast<float*>(ws + fd_states_bytes(p, batch));
  float* dp = p.P > 0 ? dparams : nullptr;
  float* dx = p.F > 0 ? dinputs : nullptr;
  float* rows = (c->shared && dp) ? reinterpret_cast<float*>(ws + fd_rows_bytes(p, batch)) : nullptr;
  if (p.path == VQC_PATH_STREAM) {
    // one forward over the shifted copies of each chunk of slots, then its
    // differences
    for (int base = 0; base < NS; base += chunk) {
      const int cs = std::min(chunk, NS - base);
      const int64_t vb = batch * 2 * cs;
      if ((rc = stream_forward(c, vb, params, inputs, ev, ws, stream, false, nullptr, nullptr,
                               base, cs,
                               h)))
        return rc;
      rc = vqc::launch_fd_combine(batch, cs, base, p.P, p.F, p.n, h, ev, grad_out,
                                  rows ? rows : dp, dx, stream);
      if (rc) return hip_fail("difference launch", rc);
    }
    if (rows && (rc = vqc::launch_sum_rows(batch, p.P, rows, dp, stream)))
      return hip_fail("parameter gradient sum", rc);
    return VQC_OK;
  }
  vqc::TileArgs a = tile_args(c, false, virt);
  a.params = params;
  a.inputs = inputs;
  a.expvals = ev;
  a.fd_slots = NS;
  a.fd_h = h;
  rc = c->engine == VQC_ENGINE_JIT
           ? vqc::jit_launch(c->jit.res_fwd, resident_blocks(p, virt), p.WG, &a, sizeof(a), stream)
           : vqc::launch_resident_forward(p, a, resident_blocks(p, virt), stream);
  if (rc) return hip_fail("shifted forward launch", rc);
  rc = vqc::launch_fd_combine(batch, NS, 0, p.P, p.F, p.n, h, ev, grad_out, rows ? rows : dp, dx,
                              stream);
  if (rc) return hip_fail("difference launch", rc);
  if (rows && (rc = vqc::launch_sum_rows(batch, p.P, rows, dp, stream)))
    return hip_fail("parameter gradient sum", rc);
  return VQC_OK;
}

int vqc_loss_grad(int32_t kind, int64_t batch, int32_t n_qubits, const float* expvals,
                  const float* target, float* grad_out, void* stream) {
  if (kind < VQC_LOSS_SUM || kind > VQC_LOSS_MSE_MEANZ)
    return fail(VQC_ERR_INVALID_ARG, "unknown loss kind");
  if (batch < 0 || n_qubits < 1 || n_qubits > VQC_MAX_QUBITS)
    return fail(VQC_ERR_INVALID_ARG, "bad batch or n_qubits");
  if (batch == 0) return VQC_OK;
  if (batch > (int64_t)INT_MAX * 256) return fail(VQC_ERR_TOO_LARGE, "batch too large");
  if (!expvals || !grad_out) return fail(VQC_ERR_INVALID_ARG, "expvals or grad_out is NULL");
  if ((kind == VQC_LOSS_MSE_Z0 || kind == VQC_LOSS_MSE_MEANZ) && !target)
    return fail(VQC_ERR_INVALID_ARG, "MSE losses need a target");
  int rc = vqc::launch_loss_grad(kind, batch, batch, n_qubits, expvals, target, grad_out, stream);
  if (rc) return fail(VQC_ERR_HIP, std::string("loss launch failed: ") +
                                       hipGetErrorString((hipError_t)rc));
  return VQC_OK;
}

int vqc_circuit_info(const vqc_circuit* c, vqc_info* info) {
  if (!c || !info) return fail(VQC_ERR_INVALID_ARG, "NULL argument");
  std::memset(info, 0, sizeof(*info));
  const Plan& p = c->plan;
  info->n_qubits = p.n;
  info->n_params = p.P;
  info->n_inputs = p.F;
  info->n_ops = p.n_ops;
  info->n_rotations = (int32_t)p.occ_src.size();
  info->path = p.path;
  info->tile_qubits = p.k;
  info->threads = p.WG;
  info->fwd_passes = p.path == VQC_PATH_STREAM ? (int32_t)p.fpass.size() : 1;
  info->bwd_passes = p.path == VQC_PATH_STREAM ? (int32_t)p.bpass.size() : 1;
  info->fwd_exchanges = p.fwd_exchanges;
  info->bwd_exchanges = p.bwd_exchanges;
  info->fwd_instructions = (int32_t)(p.fwd.size() / 2);
  info->bwd_instructions = (int32_t)(p.bwd.size() / 2);
  info->lds_bytes_fwd = (int32_t)p.lds_fwd;
  info->lds_bytes_bwd = (int32_t)p.lds_bwd;
  info->engine = c->engine;
  info->shared_params = c->shared ? 1 : 0;
  if (c->step) {
    const Plan& s = c->step->plan;
    for (const auto& hq : s.head) info->step_head_rotations += (int32_t)hq.size();
    info->step_fwd_passes = (int32_t)s.fpass.size();
    info->step_bwd_passes = (int32_t)s.bpass.size();
  }
  return VQC_OK;
}

int vqc_jit_check(const vqc_circuit* c) {
  if (!c) return fail(VQC_ERR_INVALID_ARG, "circuit handle is NULL");
  std::string log;
  int rc = vqc::jit_compile_only(c->plan, log);
  if (!rc && c->step) rc = vqc::jit_compile_only(c->step->plan, log);
  if (rc) return fail(rc, "run-time compilation failed: " + log.substr(0, 4000));
  return VQC_OK;
}

}  // extern "C"
