// api.cpp -- the C ABI declared in include/vqc.h.
#include <hip/hip_runtime_api.h>

#include <climits>
#include <cstring>
#include <new>
#include <string>

#include "vqc.h"
#include "vqc_internal.h"

using vqc::Plan;

struct vqc_circuit {
  Plan plan;
  int device = -1;   // -1: host-only plan
  void* blob = nullptr;
  size_t off_fwd = 0, off_bwd = 0, off_cols = 0, off_src = 0, off_idx = 0, off_slot = 0,
         off_cs = 0, off_end = 0;
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
  return (size_t)resident_blocks(p, batch) * (size_t)p.WG * vqc::kRegAmps * 8;
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
  a.occ_slot = at<int32_t>(c, c->off_slot);
  a.end_phys = at<uint8_t>(c, c->off_end);
  a.n_occ = (int32_t)p.occ_src.size();
  a.n_slots = p.P + p.F;
  a.P = p.P;
  a.F = p.F;
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
  if (resident_blocks(c->plan, batch) > (int64_t)INT_MAX)
    return fail(VQC_ERR_TOO_LARGE, "batch too large for one launch");
  return VQC_OK;
}

int check_rows(const vqc_circuit* c, const float* params, const float* inputs) {
  if (c->plan.P > 0 && !params) return fail(VQC_ERR_INVALID_ARG, "params is NULL but P > 0");
  if (c->plan.F > 0 && !inputs) return fail(VQC_ERR_INVALID_ARG, "inputs is NULL but F > 0");
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
  int device = 0, path = VQC_PATH_AUTO;
  if (opts) {
    for (int r : opts->reserved)
      if (r != 0) return fail(VQC_ERR_INVALID_ARG, "reserved option fields must be zero");
    device = opts->device;
    path = opts->path;
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
    h.w0 = o.wires[0];
    h.w1 = o.wires[1];
    for (int s = 0; s < 3; ++s) {
      h.src[s] = o.src[s];
      h.idx[s] = o.idx[s];
      h.val[s] = o.val[s];
    }
  }
  vqc_circuit* c = new (std::nothrow) vqc_circuit();
  if (!c) return fail(VQC_ERR_OOM, "out of host memory");
  std::string msg;
  int rc = vqc::build_plan(hops, n_qubits, n_params, n_inputs, path, c->plan, msg);
  if (rc != 0) {
    delete c;
    return fail(rc, msg);
  }
  c->device = device;
  if (device >= 0) {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device >= count) {
      delete c;
      return fail(VQC_ERR_INVALID_ARG, "no HIP device " + std::to_string(device));
    }
    const Plan& p = c->plan;
    std::vector<unsigned char> blob;
    c->off_fwd = append(blob, p.fwd);
    c->off_bwd = append(blob, p.bwd);
    c->off_cols = append(blob, p.cols);
    c->off_src = append(blob, p.occ_src);
    c->off_idx = append(blob, p.occ_idx);
    c->off_slot = append(blob, p.occ_slot);
    c->off_cs = append(blob, p.occ_cs);
    c->off_end = append(blob, p.end_phys);
    DeviceGuard g(device);
    if (!g.ok()) {
      delete c;
      return fail(VQC_ERR_HIP, "hipSetDevice failed");
    }
    if (hipMalloc(&c->blob, blob.size()) != hipSuccess) {
      delete c;
      return fail(VQC_ERR_HIP, "hipMalloc of the schedule failed");
    }
    if (hipMemcpy(c->blob, blob.data(), blob.size(), hipMemcpyHostToDevice) != hipSuccess) {
      (void)hipFree(c->blob);
      delete c;
      return fail(VQC_ERR_HIP, "copy of the schedule failed");
    }
    rc = vqc::prepare_kernels(p.WG, p.lds_fwd, p.lds_bwd);
    if (rc != 0) {
      (void)hipFree(c->blob);
      delete c;
      return fail(VQC_ERR_HIP, std::string("hipFuncSetAttribute failed: ") +
                                   hipGetErrorString((hipError_t)rc));
    }
  }
  *out = c;
  return VQC_OK;
}

void vqc_destroy(vqc_circuit* c) {
  if (!c) return;
  if (c->blob) {
    DeviceGuard g(c->device);
    (void)hipFree(c->blob);
  }
  delete c;
}

size_t vqc_workspace_bytes(const vqc_circuit* c, int64_t batch, int32_t training) {
  if (!c || batch < 0) return (size_t)-1;
  if (!training || batch == 0) return 0;
  return resident_state_bytes(c->plan, batch);
}

int vqc_forward(const vqc_circuit* c, int64_t batch, const float* params, const float* inputs,
                float* expvals, void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_runnable(c);
  if (rc) return rc;
  if ((rc = check_batch(c, batch))) return rc;
  if (batch == 0) return VQC_OK;
  if ((rc = check_rows(c, params, inputs))) return rc;
  if (!expvals) return fail(VQC_ERR_INVALID_ARG, "expvals is NULL");
  if (workspace) {
    if (workspace_bytes < resident_state_bytes(c->plan, batch))
      return fail(VQC_ERR_WORKSPACE, "workspace smaller than vqc_workspace_bytes(c, batch, 1)");
    if (reinterpret_cast<uintptr_t>(workspace) % 16)
      return fail(VQC_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  }
  DeviceGuard g(c->device);
  if (!g.ok()) return fail(VQC_ERR_HIP, "hipSetDevice failed");
  vqc::TileArgs a = tile_args(c, false, batch);
  a.params = params;
  a.inputs = inputs;
  a.expvals = expvals;
  a.ws = workspace;
  rc = vqc::launch_resident_forward(c->plan, a, resident_blocks(c->plan, batch), stream);
  if (rc) return fail(VQC_ERR_HIP, std::string("forward launch failed: ") +
                                       hipGetErrorString((hipError_t)rc));
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
  if (!workspace || workspace_bytes < resident_state_bytes(c->plan, batch))
    return fail(VQC_ERR_WORKSPACE, "backward needs the workspace of a training forward");
  if (reinterpret_cast<uintptr_t>(workspace) % 16)
    return fail(VQC_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  DeviceGuard g(c->device);
  if (!g.ok()) return fail(VQC_ERR_HIP, "hipSetDevice failed");
  vqc::TileArgs a = tile_args(c, true, batch);
  a.params = params;
  a.inputs = inputs;
  a.ws = workspace;
  a.grad_out = grad_out;
  a.dparams = c->plan.P > 0 ? dparams : nullptr;
  a.dinputs = c->plan.F > 0 ? dinputs : nullptr;
  rc = vqc::launch_resident_backward(c->plan, a, resident_blocks(c->plan, batch), stream);
  if (rc) return fail(VQC_ERR_HIP, std::string("backward launch failed: ") +
                                       hipGetErrorString((hipError_t)rc));
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
  int rc = vqc::launch_loss_grad(kind, batch, n_qubits, expvals, target, grad_out, stream);
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
  info->fwd_passes = 1;
  info->bwd_passes = 1;
  info->fwd_exchanges = p.fwd_exchanges;
  info->bwd_exchanges = p.bwd_exchanges;
  info->fwd_instructions = (int32_t)(p.fwd.size() / 2);
  info->bwd_instructions = (int32_t)(p.bwd.size() / 2);
  info->lds_bytes_fwd = (int32_t)p.lds_fwd;
  info->lds_bytes_bwd = (int32_t)p.lds_bwd;
  return VQC_OK;
}

}  // extern "C"
