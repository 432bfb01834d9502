// vqc_structs.h -- constants, instruction encoding and kernel argument records
// shared by the host library, the precompiled kernels and the kernels compiled
// at run time for a specific circuit.  Plain C++ with no standard-library
// dependency beyond <stdint.h>, so the run-time compiler can include it.
#pragma once
#ifndef __HIPCC_RTC__
#include <stddef.h>
#include <stdint.h>
#else
// the run-time compiler has no C headers: take the types from the compiler
typedef __INT32_TYPE__ int32_t;
typedef __UINT32_TYPE__ uint32_t;
typedef __INT64_TYPE__ int64_t;
typedef __UINT64_TYPE__ uint64_t;
typedef __UINT8_TYPE__ uint8_t;
typedef __INT16_TYPE__ int16_t;
typedef __UINT16_TYPE__ uint16_t;
typedef __SIZE_TYPE__ size_t;
#endif

namespace vqc {

constexpr int kDefaultRegBits = 4;           // R of the resident kernels
constexpr int kStreamRegBitsFwd = 4;         // streaming forward: 1024 threads x 16
constexpr int kStreamRegBitsBwd = 4;         // streaming adjoint: 1024 threads x 16
constexpr int kMaxTileQubits = 14;           // 2^14 c64 = 128 KiB per tile
constexpr int kMaxQubits = 20;
constexpr int kLdsBytes = 160 * 1024;        // gfx950 LDS per workgroup
constexpr int kBankBits = 5;                 // lane bits kept bank-conflict free
constexpr int kSrcParam = 0;                 // angle sources, as in the C ABI
constexpr int kSrcInput = 1;
constexpr int kSrcConst = 2;
constexpr int kLossSum = 0;                  // loss heads, as in the C ABI
constexpr int kLossMean = 1;
constexpr int kLossMseZ0 = 2;
constexpr int kLossMseMeanZ = 3;

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
  PF_LAST_ADJ = 8,    // (adjoint) the last pass: psi and lambda are not stored
};

// Arguments of the resident kernels (one launch, whole sample on chip).
struct TileArgs {
  const uint32_t* ins;      // instruction pairs (word0, arg)
  int32_t n_ins;
  const uint32_t* cols;     // exchange column tables
  const int32_t* occ_src;   // per occurrence: 0 param, 1 input, 2 const
  const int32_t* occ_idx;
  const float* occ_cs;      // per occurrence (cos, sin) of const angles / 2
  const float* occ_ma;      // per occurrence (mul, add): angle = mul * value + add;
                            // null when every occurrence is (1, 0)
  const uint8_t* end_phys;  // per logical qubit: physical bit at forward end
  // the circuit's trailing entanglers, folded into the measurement (null when
  // it has none): per measured qubit the logical Z-string whose expectation is
  // its <Z>, and per qubit the image of its basis-index bit (probabilities)
  const uint32_t* zmask;
  const uint32_t* pcol;
  int32_t n_occ, n_slots, P, F;
  int32_t pstride;          // row stride of params: P, or 0 when shared by the batch
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
  // training step only (forward, loss head and adjoint in one launch)
  const uint32_t* ins_b;    // the adjoint's instruction pairs
  int32_t n_ins_b;
  int32_t loss;             // loss head kLoss*
  const float* target;      // [B] (MSE heads)
  float* cot_out;           // [B, n] cotangent written here when not null
  uint32_t lds_e;           // byte offset of E and g rows [S][n] each
  // central differences (forward only): B counts shifted copies, 2 per slot
  int32_t fd_slots;         // P + F, or 0
  float fd_h;
  // forward only: initial states and basis-state probabilities (logical order)
  const void* psi0;         // float2 [B][2^n] initial states, or null for |0...0>
  const uint8_t* start_phys;  // per logical qubit: physical bit at forward start
  float* probs;             // [B][2^n] |psi_x|^2 of the final states, or null
};

// Arguments of one streaming pass (one 2^k tile per workgroup, k <= 14).
struct PassArgs {
  const uint32_t* ins;
  int32_t n_ins;
  const uint32_t* cols;
  const uint32_t* io;          // tile I/O columns (k + ng): loads, in the layout read
  const uint32_t* io_out;      // stores, in the layout written
  const uint32_t* io_lin;      // loads in logical order (Psi_0)
  const uint32_t* io_lout;     // stores in logical order (probabilities)
  const uint8_t* start_phys;   // logical -> phys at pass start
  const uint8_t* end_phys;     // logical -> phys at pass end
  const uint32_t* zmask;       // measured Z-strings (as in TileArgs), or null
  const int32_t* pslots;       // pass-local -> global gradient slot
  int32_t n_pslots;
  int32_t flags;
  int32_t psi0_in;             // 1: this (first forward) pass reads Psi_0, logical order
  const int32_t* occ_src;
  const int32_t* occ_idx;
  const float* occ_cs;
  const float* occ_ma;         // (mul, add) per occurrence, or null
  int32_t n_occ, n_slots, P, F, n, k, ng;
  int32_t pstride;             // row stride of params: P, or 0 when shared by the batch
  int64_t B;
  const float* params;
  const float* inputs;
  const void* psi_src;        // float2 states [B][2^n] in the pass's input / output
                               // memory layouts (Psi_0: logical order)
  void* psi_dst;
  const void* lam_src;
  void* lam_dst;
  float* epart;                // [B * 2^ng, n] <Z> partial sums
  float* gpart;                // [B * 2^ng, n_slots] gradient partial sums
  const float* grad_out;
  uint32_t lds_tab, lds_acc;
  float* probs;                // (last forward pass) [B][2^n] probabilities, or null
  // central differences: B counts shifted copies, 2 per slot of the chunk
  int32_t fd_slots, fd_base;   // slots fd_base .. fd_base + fd_slots - 1, or fd_slots 0
  float fd_h;
  // per-sample tables of the generated kernels' tangent form, written once per
  // call by the table kernel and read by every pass: (t, cos phi') pairs
  // [B][n_occ][2], the adjoint's gradient signs [B][n_occ], the <Z> signs [B][n]
  float* tabs;
  float* gsig;
  float* esig;
  // training step with a product head: per tile of the last adjoint pass the
  // partial sums of the 2-vectors v_q [B * 2^ng][NV] (NV = 4 n rounded up to 16),
  // and the gradient rows the head kernel writes (dparams [B][P] or null,
  // dinputs [B][F] or null)
  float* vpart;
  float* dparams;
  float* dinputs;
};
}  // namespace vqc
