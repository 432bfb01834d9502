// vqc_internal.h -- schedule format shared by the host planner and the gfx950
// kernels (not part of the public ABI).
//
// Execution model ("register tile").  A workgroup holds a tile of 2^k
// amplitudes of one sample (or several small samples) entirely on chip:
//   physical bit p of an amplitude's tile position
//     p in [0, R)      -> register index j of the owning thread (2^R amps/thread)
//     p in [R, k)      -> bit (p - R) of the thread index within the tile
// A mapping phys -> logical qubit says which qubit every physical bit holds.
// Non-diagonal gates (RX, RY, CNOT target) act on a register bit and are pure
// VALU work; diagonal gates (RZ, CZ) and CNOT controls act wherever the qubit
// sits.  An EXCHANGE instruction permutes the tile through LDS so that other
// qubits land on register bits (compile-time planned, Belady order).  The
// schedule is a uniform instruction stream read with scalar loads.
#pragma once
#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "vqc_structs.h"

namespace vqc {

struct PassPlan {
  int ins_off = 0, n_ins = 0;   // instruction pairs (offset in pairs)
  // tile I/O columns, k + ng words each: the address bit of each tile rank bit
  // (thread bits, then register bits), then of each global bit
  int io_off = 0;               // loads, in the memory layout the pass reads
  int io_out_off = 0;           // stores, in the layout it writes
  int io_lin_off = 0;           // loads in logical order (Psi_0)
  int io_lout_off = 0;          // stores in logical order (probabilities)
  int start_off = 0, end_off = 0;  // nq bytes each: logical qubit -> physical bit
  int slots_off = 0, n_slots = 0;  // pass-local gradient slot -> global slot
  int flags = 0;
};

struct Prim {
  int kind;
  int q0, q1;  // target (1q) / control,target (CNOT) / a,b (CZ)
  int occ;     // angle occurrence index for rotations, -1 otherwise
};

struct Plan {
  int n = 0, nq = 0, k = 0, t = 0, WG = 0, S = 0, G = 0;
  int R = kDefaultRegBits;                // register bits of the resident kernels
  int Rf = kStreamRegBitsFwd, Rb = kStreamRegBitsBwd;  // streaming forward / adjoint
  int ng = 0;                             // global (streamed) qubits
  int lanes = 0;                          // lane bits that take RX / RY / CNOT targets
  int P = 0, F = 0, n_ops = 0, path = 1;
  std::vector<Prim> prims;
  // Trailing entanglers (CNOT / CZ with no later rotation on their qubits) are
  // not run: <Z_j> after them is the expectation of the Z-string zmask[j]
  // before them, and a basis state x before them is A x after them, A the
  // GF(2) map with columns pcol[q].  Both empty when there are none.
  std::vector<Prim> tail;
  std::vector<uint32_t> zmask, pcol;
  // Each qubit's head: the rotations on it before any entangler touches it, in
  // circuit order.  The state after every head is a product state, which the
  // generated training step builds directly (and whose gradients it takes from
  // lambda contracted against the other qubits' states).
  std::vector<std::vector<Prim>> head;
  // Streaming training step plan: prims leave out the heads' rotations (the
  // first forward pass starts from the product state after them).
  bool product_head = false;
  std::vector<int32_t> occ_src, occ_idx, occ_slot;
  std::vector<float> occ_cs;              // 2 per occurrence
  std::vector<float> occ_ma;              // 2 per occurrence: angle = mul * value + add
  bool affine = false;                    // some occurrence has (mul, add) != (1, 0)
  double const_drift = 0.0;               // sum of the constants' cos^2 + sin^2 - 1 (planning)
  std::vector<uint32_t> fwd, bwd;         // instruction pairs
  std::vector<uint32_t> cols;             // exchange / tile I/O column tables
  std::vector<uint8_t> maps;              // logical -> phys tables (nq bytes each)
  std::vector<int32_t> pslots;            // pass-local -> global gradient slots
  std::vector<PassPlan> fpass, bpass;     // streaming passes
  int start_off = 0, end_off = 0;         // resident: forward start / end mapping in `maps`
  int bwd_end_off = 0;                    // resident: the adjoint's end mapping in `maps`
  int fwd_exchanges = 0, bwd_exchanges = 0;
  int max_pass_slots = 0;
  size_t lds_fwd = 0, lds_bwd = 0, lds_tab = 0, lds_acc = 0;
  size_t lds_e = 0, lds_step = 0;  // resident training step (0 when streaming)
};

// Host planning (no device calls).  Returns 0 or a VQC_ERR_* code with msg.
struct HostOp {
  int32_t kind, w[3];
  int32_t src[3], idx[3];
  float val[3], mul[3];
};
constexpr int kNumGateKinds = 32;  // VQC_RX .. VQC_CSWAP
// lane_gates: the schedule may put RX / RY / CNOT targets on lane bits (only
// the generated kernels run such schedules).
// tile_qubits: streaming tile size (0 = default).
int build_plan(const std::vector<HostOp>& ops, int n, int P, int F, int path, int reg_bits,
               Plan& plan, std::string& msg, bool lane_gates, int tile_qubits = 0);
// Gradient slots (P + F) up to which the streaming training step runs a plan
// without the heads (its head kernel holds a row of them in LDS).
constexpr int kMaxStepSlots = 8192;
// The streaming training step's plan without the heads' rotations (planner.cpp).
// Returns 0, 1 when the circuit has no head rotation, or a VQC_ERR_* code.
int build_step_plan(const Plan& full, Plan& step, std::string& msg);
// OpenQASM front end (qasm.cpp).  Returns 0 or a VQC_ERR_* code with msg.
int parse_qasm(const char* source, const char* input_names, std::vector<vqc_op>& ops,
               int& n_qubits, int& n_params, int& n_inputs, std::string& msg);

// Kernel launchers (kernels.hip).  Return 0 or a hipError_t value.
int launch_resident_forward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream);
int launch_resident_backward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream);
int launch_resident_step(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream);

int launch_stream_pass(const Plan& plan, bool bwd, const PassArgs& a, int64_t blocks,
                       void* stream);
int launch_reduce_e(int64_t batch, int ng, int n, const float* epart, float* e, void* stream);
// <Z> rows and the loss head's cotangent rows of `batch` rows of a batch of
// `norm` samples in one launch (n <= 256)
int launch_reduce_e_loss(int64_t batch, int ng, int n, const float* epart, float* e, int kind,
                         int64_t norm, const float* y, float* g, void* stream);
int launch_reduce_grad(int64_t batch, int ng, int n_slots, int P, int F, const float* gpart,
                       float* dparams, float* dinputs, void* stream);
int launch_fill_zero(float* p, int64_t count, void* stream);
// slots base .. base + NS - 1 of the central differences; ev [batch][NS][2][n]
int launch_fd_combine(int64_t batch, int NS, int base, int P, int F, int n, float h,
                      const float* ev, const float* g, float* dparams, float* dinputs,
                      void* stream);
// out[p] = sum over b of rows[b * P + p], in a fixed order
int launch_sum_rows(int64_t batch, int P, const float* rows, float* out, void* stream);
// rows [0, batch) of a batch of `norm` samples (the MSE losses divide by norm)
int launch_loss_grad(int kind, int64_t batch, int64_t norm, int n, const float* e, const float* y,
                     float* g, void* stream);
// Device address of the static scratch array (VQC_NOALLOC_SCRATCH_BYTES) on
// `device`, which must be the current device; looked up once per device and
// kept.  Returns 0 or a hipError_t value.
constexpr int kScratchDevices = 64;
int scratch_pointer(int device, void** out);
int prepare_kernels(const Plan& plan);

// Kernels compiled at run time for one circuit (jit.cpp).
struct JitKernels {
  void* res_fwd = nullptr;            // hipFunction_t
  void* res_bwd = nullptr;
  void* res_step = nullptr;           // forward, loss head and adjoint in one launch
  std::vector<void*> pass_fwd, pass_bwd;
  void* tables = nullptr;             // streaming: the per-sample table kernel, or none
  void* head_finish = nullptr;        // streaming step with a product head: head gradients
};
constexpr int kTableThreads = 256;    // threads of the table kernel's workgroups
// threads of the streaming step's head kernel (one workgroup per sample: its
// sums over the tiles of every gradient slot are spread over them)
constexpr int kHeadThreads = 256;
struct JitUnit {
  std::string name, src;
  // what the kernel is: resident forward / adjoint / step ('r', 'b', 's'),
  // streaming forward pass / adjoint pass / tables / head gradients ('F', 'B', 'T', 'G')
  char role;
};
std::vector<JitUnit> jit_units(const Plan& plan);
bool stream_tables_fit(const Plan& plan);
int jit_compile_only(const Plan& plan, std::string& log);
// hiprtc compilation of one generated kernel (jit_compile.cpp)
int compile_source(const std::string& src, std::vector<char>& code, std::string& log);
int jit_build(const Plan& plan, int device, JitKernels& out, std::string& msg);
int jit_launch(void* fn, int64_t blocks, int threads, const void* args, size_t args_size,
               void* stream);

}  // namespace vqc
