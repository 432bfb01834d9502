// vqc_internal.h -- schedule format shared by the host planner and the gfx950
// kernels (not part of the public ABI).
//
// Execution model ("register tile").  A workgroup holds a tile of 2^k
// amplitudes of one sample (or several small samples) entirely on chip:
//   physical bit p of an amplitude's tile position
//     p in [0, R)      -> register index j of the owning thread (16 amps/thread)
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

namespace vqc {

constexpr int kRegBits = 4;                  // R: register bits per thread
constexpr int kRegAmps = 1 << kRegBits;      // amplitudes per thread
constexpr int kMaxTileQubits = 14;           // 2^14 c64 = 128 KiB per tile
constexpr int kMaxQubits = 20;
constexpr int kLdsBytes = 160 * 1024;        // gfx950 LDS per workgroup
constexpr int kBankBits = 5;                 // lane bits kept bank-conflict free

// primitive kinds after lowering (ROT -> RZ, RY, RZ)
enum PrimKind : int { P_RX = 0, P_RY = 1, P_RZ = 2, P_CNOT = 4, P_CZ = 5 };

// instruction opcodes.  Physical bits p >= k name global qubits of a
// streamed tile (bit p - k of the tile index within the sample).
enum Opcode : uint32_t {
  OP_RX = 1,      // a = register position, arg = occurrence
  OP_RY = 2,      // a = register position, arg = occurrence
  OP_RZ = 3,      // a = physical bit,      arg = occurrence
  OP_CNOT = 4,    // a = control physical bit, b = target register position
  OP_CZ = 5,      // a, b = physical bits
  OP_EXCHANGE = 6 // arg = offset of 2k column words (write side, read side)
};

// word0 = op | a << 5 | b << 10 | (slot + 1) << 16; word1 = arg.  `slot` is the
// gradient accumulator of a rotation (-1: constant angle, no gradient).
inline uint32_t ins_word0(uint32_t op, uint32_t a, uint32_t b, int slot) {
  return op | (a << 5) | (b << 10) | ((uint32_t)(slot + 1) << 16);
}

// pass flags of the streaming kernels
enum PassFlag : int32_t {
  PF_INIT = 1,        // start from |0...0> instead of loading psi
  PF_MAKE_LAMBDA = 2, // (adjoint) lambda = H psi after loading psi_G
  PF_ZPART = 4,       // (forward) per-tile <Z> partial sums
};

struct PassPlan {
  int ins_off = 0, n_ins = 0;   // instruction pairs (offset in pairs)
  int io_off = 0;               // k + ng words: x offset of each tile rank bit, then
                                // of each global bit
  int start_off = 0, end_off = 0;  // nq bytes each: logical qubit -> physical bit
  int slots_off = 0, n_slots = 0;  // pass-local gradient slot -> global slot
  int flags = 0;
};

struct Prim {
  int kind;
  int q0, q1;  // target (1q) / control,target (CNOT) / a,b (CZ)
  int occ;     // angle occurrence index for rotations, -1 otherwise
};

// Arguments of the resident kernels (one launch, whole sample on chip).
struct TileArgs {
  const uint32_t* ins;      // instruction pairs (word0, arg)
  int32_t n_ins;
  const uint32_t* cols;     // exchange column tables
  const int32_t* occ_src;   // per occurrence: 0 param, 1 input, 2 const
  const int32_t* occ_idx;
  const float* occ_cs;      // per occurrence (cos, sin) of const angles / 2
  const uint8_t* end_phys;  // per logical qubit: physical bit at forward end
  int32_t n_occ, n_slots, P, F;
  int32_t n;                // real qubits (E and g have n columns)
  int32_t k;                // tile qubits (>= 4)
  int32_t t;                // thread bits per sample: k - R
  int32_t S;                // samples per workgroup
  int32_t G;                // reduction groups per workgroup
  int64_t B;
  const float* params;
  const float* inputs;
  float* expvals;
  void* ws;                 // saved final states (training) or null
  const float* grad_out;
  float* dparams;
  float* dinputs;
  uint32_t lds_tab;         // byte offset of the angle table in LDS
  uint32_t lds_acc;         // byte offset of the gradient accumulators
};

struct Plan {
  int n = 0, nq = 0, k = 0, t = 0, WG = 0, S = 0, G = 0;
  int ng = 0;                             // global (streamed) qubits
  int P = 0, F = 0, n_ops = 0, path = 1;
  std::vector<Prim> prims;
  std::vector<int32_t> occ_src, occ_idx, occ_slot;
  std::vector<float> occ_cs;              // 2 per occurrence
  std::vector<uint32_t> fwd, bwd;         // instruction pairs
  std::vector<uint32_t> cols;             // exchange / tile I/O column tables
  std::vector<uint8_t> maps;              // logical -> phys tables (nq bytes each)
  std::vector<int32_t> pslots;            // pass-local -> global gradient slots
  std::vector<PassPlan> fpass, bpass;     // streaming passes
  int end_off = 0;                        // resident: forward end mapping in `maps`
  int fwd_exchanges = 0, bwd_exchanges = 0;
  int max_pass_slots = 0;
  size_t lds_fwd = 0, lds_bwd = 0, lds_tab = 0, lds_acc = 0;
};

// Host planning (no device calls).  Returns 0 or a VQC_ERR_* code with msg.
struct HostOp {
  int32_t kind, w0, w1;
  int32_t src[3], idx[3];
  float val[3];
};
int build_plan(const std::vector<HostOp>& ops, int n, int P, int F, int path, Plan& plan,
               std::string& msg);

// Kernel launchers (kernels.hip).  Return 0 or a hipError_t value.
int launch_resident_forward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream);
int launch_resident_backward(const Plan& plan, const TileArgs& a, int64_t blocks, void* stream);

// Arguments of one streaming pass (1024 threads, one 2^14 tile per workgroup).
struct PassArgs {
  const uint32_t* ins;
  int32_t n_ins;
  const uint32_t* cols;
  const uint32_t* io;          // tile I/O columns (k + ng)
  const uint8_t* start_phys;   // logical -> phys at pass start
  const uint8_t* end_phys;     // logical -> phys at pass end
  const int32_t* pslots;       // pass-local -> global gradient slot
  int32_t n_pslots;
  int32_t flags;
  const int32_t* occ_src;
  const int32_t* occ_idx;
  const float* occ_cs;
  int32_t n_occ, n_slots, P, F, n, k, ng;
  int64_t B;
  const float* params;
  const float* inputs;
  const void* psi_src;        // float2 states, logical order [B][2^n]
  void* psi_dst;
  const void* lam_src;
  void* lam_dst;
  float* epart;                // [B * 2^ng, n] <Z> partial sums
  float* gpart;                // [B * 2^ng, n_slots] gradient partial sums
  const float* grad_out;
  uint32_t lds_tab, lds_acc;
};
int launch_stream_pass(bool bwd, const PassArgs& a, int64_t blocks, size_t lds, void* stream);
int launch_reduce_e(int64_t batch, int ng, int n, const float* epart, float* e, void* stream);
int launch_reduce_grad(int64_t batch, int ng, int n_slots, int P, int F, const float* gpart,
                       float* dparams, float* dinputs, void* stream);
int launch_fill_zero(float* p, int64_t count, void* stream);
int prepare_stream_kernels(size_t lds_fwd, size_t lds_bwd);
int launch_loss_grad(int kind, int64_t batch, int n, const float* e, const float* y, float* g,
                     void* stream);
int prepare_kernels(int wg, size_t lds_fwd, size_t lds_bwd);

}  // namespace vqc
