/*
 * vqc.h -- C ABI of the batched VQC statevector engine for MI355X (gfx950).
 *
 * The library runs the execute phase of compile-once VQC simulation on the GPU:
 * a static parametrized circuit over the standard gate library (Pauli
 * rotations, ROT, U3, the fixed Clifford+T gates, controlled and two-qubit
 * rotations, SWAP, CCX, CSWAP) is compiled once into a device schedule (Sec. 3
 * "Compile-Once Lowering and Execution"; Algorithm 1, compile phase) and then
 * applied to B independent 2^n-amplitude complex64 states, each starting in
 * |0...0> or a given Psi_0 (Algorithm 1, execute phase).  vqc_compile_qasm
 * takes the circuit as OpenQASM text.  The forward pass returns the per-qubit
 * Pauli-Z expectations E[b, j] = sum_x (-1)^{x_j} |psi_b[x]|^2 (Algorithm 1,
 * return statement).  The backward pass returns the exact gradient of
 * L_b = sum_j g[b, j] E[b, j] with respect to every per-sample parameter and
 * encoded input (Sec. 3 "Gate Application and Differentiation"), computed by
 * the adjoint method instead of a stored tape.
 *
 * Conventions shared by every entry point
 *   - Rotations are R_P(t) = exp(-i t P / 2); ROT(phi, theta, omega) is
 *     RZ(omega) RY(theta) RZ(phi) with phi applied first.  Qubit j is bit j of
 *     the basis index.  CNOT(c, t) flips t when c is 1; CZ(a, b) negates the
 *     amplitudes with both bits set.  The other gates are the OpenQASM standard
 *     library's: P(l) = diag(1, e^{il}); U3(t, p, l) = [[c, -e^{il} s],
 *     [e^{ip} s, e^{i(p+l)} c]] (c, s of t/2); U2(p, l) = U3(pi/2, p, l); H, S,
 *     SDG, T, TDG, SX = sqrt(X), SXDG, X, Y, Z, ID; controlled gates (control =
 *     wires[0]) act on the target when the control is 1; R_PP(t) =
 *     exp(-i t P(x)P / 2); CCX(c0, c1, t); CSWAP(c, a, b).  Every gate is
 *     applied up to a global phase, which no output depends on.
 *   - Device arrays are fp32, row-major, contiguous, device-resident and owned
 *     by the caller; the library never allocates or frees them.  Outputs are
 *     overwritten, never accumulated.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *     enqueue work and return; launch failures return VQC_ERR_HIP, faults
 *     inside kernels surface at the caller's next synchronisation.
 *   - Every function returns VQC_OK (0) or a negative status; the message of
 *     the last failure on the calling thread is vqc_last_error().
 *   - A compiled circuit is immutable: it may be used from several threads
 *     and streams at once.
 */
#ifndef VQC_ABI_H_
#define VQC_ABI_H_

#ifndef __HIPCC_RTC__ /* the run-time compiler predefines the fixed-width types */
#include <stddef.h>
#include <stdint.h>
#endif

#ifdef __cplusplus
extern "C" {
#endif

#define VQC_MAX_QUBITS 20

/* status codes */
#define VQC_OK 0
#define VQC_ERR_INVALID_ARG -1 /* bad argument: null pointer, bad wire, bad index */
#define VQC_ERR_UNSUPPORTED -2 /* valid request the library does not support */
#define VQC_ERR_TOO_LARGE -3   /* size limits exceeded (qubits, batch, schedule) */
#define VQC_ERR_WORKSPACE -4   /* workspace missing or smaller than required */
#define VQC_ERR_HIP -5         /* a HIP runtime call failed */
#define VQC_ERR_OOM -6         /* the library's own (schedule) allocation failed */

/* gate kinds */
#define VQC_RX 0
#define VQC_RY 1
#define VQC_RZ 2
#define VQC_ROT 3
#define VQC_CNOT 4
#define VQC_CZ 5
#define VQC_ID 6
#define VQC_X 7
#define VQC_Y 8
#define VQC_Z 9
#define VQC_H 10
#define VQC_S 11
#define VQC_SDG 12
#define VQC_T 13
#define VQC_TDG 14
#define VQC_SX 15
#define VQC_SXDG 16
#define VQC_P 17     /* also OpenQASM u1 */
#define VQC_U2 18    /* (phi, lambda) */
#define VQC_U3 19    /* (theta, phi, lambda); also OpenQASM u */
#define VQC_CY 20
#define VQC_CH 21
#define VQC_SWAP 22
#define VQC_CRX 23
#define VQC_CRY 24
#define VQC_CRZ 25
#define VQC_CP 26    /* also OpenQASM cu1 */
#define VQC_RXX 27
#define VQC_RYY 28
#define VQC_RZZ 29
#define VQC_CCX 30   /* controls wires[0], wires[1]; target wires[2] */
#define VQC_CSWAP 31 /* control wires[0]; swaps wires[1], wires[2] */

/* angle sources */
#define VQC_SRC_PARAM 0 /* params[b, idx] */
#define VQC_SRC_INPUT 1 /* inputs[b, idx] */
#define VQC_SRC_CONST 2 /* val, fixed at compile time (cached, Algorithm 1 compile phase) */

/*
 * One gate of the static sequence G = {(g_i, w_i, p_i)} (Algorithm 1, compile
 * phase).  wires[0..k) are the gate's k qubits in the order of its definition
 * (one-qubit gates: the target; CNOT / controlled gates: control, target; CZ,
 * SWAP, R_PP: the two qubits; CCX: two controls, target; CSWAP: control, the
 * two swapped qubits); unused wires are ignored.  Angle slot s (RX/RY/RZ/P and
 * the controlled and two-qubit rotations: 0; ROT: phi, theta, omega; U3:
 * theta, phi, lambda; U2: phi, lambda) is
 *   src[s] == VQC_SRC_CONST:          angle = val[s]
 *   src[s] == VQC_SRC_PARAM / INPUT:  angle = mul[s] * value + val[s]
 * with value = params[b, idx[s]] or inputs[b, idx[s]]; mul[s] must be finite
 * and nonzero, and gradients carry the factor mul[s] (chain rule).
 */
typedef struct {
    int32_t kind;
    int32_t wires[3];
    int32_t src[3];
    int32_t idx[3];
    float val[3];
    float mul[3];
} vqc_op;

typedef struct vqc_circuit vqc_circuit;

/* compile options (pass NULL for the defaults) */
#define VQC_PATH_AUTO 0     /* resident for n <= 13, streaming from n = 14 (at 14
                               qubits the streaming passes were measured faster
                               than the one-launch resident step) */
#define VQC_PATH_RESIDENT 1 /* one launch, state on chip; requires n <= 14 */
#define VQC_PATH_STREAM 2   /* tiles of 2^k amplitudes (k = tile_qubits) streamed
                               through HBM, one launch per pass; n >= 14 */
#define VQC_ENGINE_JIT 0    /* kernels generated for this circuit and compiled at
                               vqc_compile time (straight-line schedule) */
#define VQC_ENGINE_INTERP 1 /* precompiled kernels that interpret the schedule */
typedef struct {
    int32_t device;      /* HIP device that receives the schedule; -1 = plan on
                            the host only (validation and introspection; the
                            handle cannot run) */
    int32_t path;        /* VQC_PATH_* */
    int32_t reg_bits;    /* amplitudes per thread = 2^reg_bits: resident path
                            2, 3 or 4 (default 4); streaming path 4 or 5 for both
                            sweeps (default: forward 4, adjoint 5); 0 = default */
    int32_t engine;      /* VQC_ENGINE_* */
    int32_t shared_params; /* 1: one parameter vector for the whole batch
                              (Algorithm 1's shared theta): params is [P] in
                              every call and dparams is [P], the sum over the
                              samples.  Inputs stay per sample.  0: per-sample
                              rows [B, P] */
    int32_t tile_qubits; /* streaming path: qubits per tile, 12, 13 or 14
                            (0 = the default: with the generated kernels 12,
                            unless its plan takes more than a quarter more
                            passes than 13, then 13; 14 with the
                            interpreter).  Each qubit less halves a
                            workgroup's LDS, so more workgroups share a CU
                            and one's HBM traffic overlaps another's compute,
                            at the cost of more passes where the circuit
                            needs them.  12 and 13: generated kernels only
                            (the interpreter runs 14) */
    int32_t reserved[2]; /* must be zero */
} vqc_compile_opts;

/*
 * vqc_compile -- validate a static gate list and build its device schedule
 * (Algorithm 1, compile phase: parse, cache constant gates, classify static
 * vs parametric).  ops: host array of n_ops gates (n_ops >= 0).  n_qubits in
 * [1, VQC_MAX_QUBITS].  n_params, n_inputs >= 0 are the row widths P and F of
 * the params/inputs arrays given at run time.  On success *out receives a
 * handle that owns only the compiled schedule (host and device copies).
 * With VQC_ENGINE_JIT (the default) and device >= 0 the kernels of this
 * circuit are generated and compiled for the device here (seconds for large
 * circuits; compiled modules are cached per process and source text).
 * Errors: VQC_ERR_INVALID_ARG (null pointer, wire out of range, a wire twice
 * in one gate, unknown kind or source, index out of range, a zero or
 * non-finite mul, a non-finite val, unknown option),
 * VQC_ERR_UNSUPPORTED (path not possible for n_qubits, run-time compilation
 * failed), VQC_ERR_TOO_LARGE (qubits or schedule beyond the limits),
 * VQC_ERR_HIP, VQC_ERR_OOM.
 */
int vqc_compile(const vqc_op *ops, int32_t n_ops, int32_t n_qubits, int32_t n_params,
                int32_t n_inputs, const vqc_compile_opts *opts, vqc_circuit **out);

/*
 * vqc_parse_qasm -- the OpenQASM front end alone (Sec. 3: a normalized
 * OpenQASM circuit is lowered once; Algorithm 1, compile phase: parse C into
 * the gate sequence).  Host only, no device.
 *   source       NUL-terminated OpenQASM 2.0, or the static subset of
 *                OpenQASM 3: qreg/qubit and creg/bit registers (qubits
 *                numbered across registers in declaration order), the
 *                standard gate library (qelib1.inc / stdgates.inc names,
 *                plus u, U, CX, cnot, phase, cphase, toffoli, fredkin),
 *                user gate definitions, register broadcasting, barrier,
 *                gphase, and terminal measurement.
 *   input_names  comma-separated names of declared inputs that are data
 *                features (inputs[b, .]); every other declared input
 *                (`input float theta;`, `input array[float[64], 8] w;`) is a
 *                trainable parameter.  Slots follow declaration order, an
 *                array taking consecutive slots.  NULL: no data inputs.
 *   Angles are expressions in numbers, pi, tau, euler, declared inputs,
 *   + - * / ^ and sin cos tan exp ln sqrt arcsin arccos arctan; each must be
 *   constant or affine in one input (then it becomes mul * value + val).
 *   ops/capacity receive the gate list (ops may be NULL with capacity 0 to
 *   query the count); *n_ops, *n_qubits, *n_params, *n_inputs are written on
 *   success even when the capacity is too small (then VQC_ERR_TOO_LARGE).
 * Errors: VQC_ERR_INVALID_ARG (syntax, unknown names, out-of-range indices,
 * non-affine angles; the message gives line:column), VQC_ERR_UNSUPPORTED
 * (reset, mid-circuit measurement, classical control, loops, subroutines,
 * gate modifiers, opaque gates, other includes, gates outside the library),
 * VQC_ERR_TOO_LARGE, VQC_ERR_OOM.
 */
int vqc_parse_qasm(const char *source, const char *input_names, vqc_op *ops, int32_t capacity,
                   int32_t *n_ops, int32_t *n_qubits, int32_t *n_params, int32_t *n_inputs);

/*
 * vqc_compile_qasm -- vqc_parse_qasm followed by vqc_compile of its gate list
 * with n_qubits, n_params and n_inputs from the program (vqc_circuit_info
 * reports them).  Errors: those of both.
 */
int vqc_compile_qasm(const char *source, const char *input_names, const vqc_compile_opts *opts,
                     vqc_circuit **out);

/* Frees the handle and its device schedule.  NULL is ignored. */
void vqc_destroy(vqc_circuit *c);

/*
 * vqc_workspace_bytes -- device workspace for `batch` samples of
 *   training = 0: an inference vqc_forward;
 *   training = 1: a training vqc_forward (the saved final states) and the
 *                 vqc_backward calls that use it (plus their scratch);
 *   training = 2: vqc_train_step;
 *   training = 3: vqc_fd_backward.
 * 0 means no workspace is needed.  Returns (size_t)-1 on invalid arguments.
 *
 * Streams.  On the streaming path (batch >= 2) vqc_forward, vqc_forward_ex,
 * vqc_backward and vqc_train_step run the first ceil(batch / 2) samples on
 * `stream` and the rest on a side stream that the library creates on the
 * device at first use (default priority) and keeps until exit: the side
 * stream waits for the work queued on `stream` before the call, and `stream`
 * waits for the side stream at its end, so each call is ordered on `stream`
 * like a single launch.  Calls that overlap on one device share the side
 * stream (they stay correct but queue behind each other there); under stream
 * capture the side stream joins the capture.  The two halves have workspace
 * layouts of their own, which vqc_workspace_bytes accounts for.
 */
size_t vqc_workspace_bytes(const vqc_circuit *c, int64_t batch, int32_t training);

/*
 * vqc_forward -- E = expectations of the circuit for `batch` samples.
 *   params   [batch, P] fp32, or [P] with shared_params (may be NULL when P == 0)
 *   inputs   [batch, F] fp32 (may be NULL when F == 0)
 *   expvals  [batch, n] fp32, written
 *   workspace / workspace_bytes: NULL/0 for inference when
 *     vqc_workspace_bytes(c, batch, 0) == 0; for training pass at least
 *     vqc_workspace_bytes(c, batch, 1) bytes, 256-byte aligned -- the final
 *     states are saved there for vqc_backward.
 * batch == 0 is a no-op.  Errors: VQC_ERR_INVALID_ARG, VQC_ERR_WORKSPACE,
 * VQC_ERR_TOO_LARGE, VQC_ERR_HIP.
 */
int vqc_forward(const vqc_circuit *c, int64_t batch, const float *params, const float *inputs,
                float *expvals, void *workspace, size_t workspace_bytes, void *stream);

/*
 * vqc_forward_ex -- vqc_forward with the execute phase's optional input and
 * its other output (Algorithm 1: the state starts from Psi_0 when one is
 * given, else |0...0>; Sec. 3: the final state yields basis-state
 * probabilities or Pauli-Z expectations).
 *   psi0    [batch, 2^n] complex64 (interleaved re, im), device, 8-byte
 *           aligned, or NULL for |0...0>.  Basis index x holds qubit q in bit
 *           q.  Used as given: it is not normalized, and the evolution is
 *           linear in it.  Read only.
 *   expvals [batch, n] fp32 written, or NULL
 *   probs   [batch, 2^n] fp32 written, or NULL: |Psi_x|^2 of the final state
 *           (they sum to |Psi_0|^2 per sample)
 * At least one of expvals, probs must be non-NULL.  params, inputs and the
 * workspace are as in vqc_forward: with a training workspace the final states
 * are saved, and vqc_backward then gives the gradients of this forward
 * (Psi_0 held fixed).  Errors: VQC_ERR_INVALID_ARG (also a misaligned psi0 or
 * probs), VQC_ERR_WORKSPACE, VQC_ERR_TOO_LARGE, VQC_ERR_HIP.
 */
int vqc_forward_ex(const vqc_circuit *c, int64_t batch, const float *params, const float *inputs,
                   const void *psi0, float *expvals, float *probs, void *workspace,
                   size_t workspace_bytes, void *stream);

/*
 * vqc_backward -- adjoint-method gradient (Sec. 3 "Gate Application and
 * Differentiation"; exact, same result as reverse-mode AD over the tape).
 *   grad_out [batch, n] fp32: cotangent g of E
 *   workspace: the one a training forward with the same circuit, batch,
 *     params and inputs filled, in stream order before this call.  The saved
 *     states are left intact (the rest is scratch), so several cotangents may
 *     be back-propagated from one forward.
 *   dparams [batch, P], dinputs [batch, F] fp32: written (per-sample
 *     gradients; a parameter used by several gates receives the sum).  Either
 *     may be NULL to skip it.  With shared_params, dparams is [P]: the sum of
 *     the samples' gradients, in a fixed order.
 * Errors: VQC_ERR_INVALID_ARG, VQC_ERR_WORKSPACE, VQC_ERR_HIP.
 */
int vqc_backward(const vqc_circuit *c, int64_t batch, const float *params, const float *inputs,
                 const float *grad_out, void *workspace, size_t workspace_bytes, float *dparams,
                 float *dinputs, void *stream);

/*
 * vqc_loss_grad -- cotangent g = dL/dE of a scalar objective over E
 * (Sec. 4.2.3: the shared objective is the mean of single-qubit <Z>):
 *   VQC_LOSS_SUM       L = sum_b sum_j E[b,j]                 g = 1
 *   VQC_LOSS_MEAN      L = sum_b mean_j E[b,j]                g = 1/n
 *   VQC_LOSS_MSE_Z0    L = mean_b (E[b,0] - y[b])^2           g[b,0] = 2(E[b,0]-y[b])/batch
 *   VQC_LOSS_MSE_MEANZ L = mean_b (mean_j E[b,j] - y[b])^2    g[b,j] = 2(s_b-y[b])/(n batch)
 * expvals [batch, n], target y [batch] (NULL for SUM/MEAN), grad_out
 * [batch, n] written.  Errors: VQC_ERR_INVALID_ARG, VQC_ERR_HIP.
 */
#define VQC_LOSS_SUM 0
#define VQC_LOSS_MEAN 1
#define VQC_LOSS_MSE_Z0 2
#define VQC_LOSS_MSE_MEANZ 3
int vqc_loss_grad(int32_t kind, int64_t batch, int32_t n_qubits, const float *expvals,
                  const float *target, float *grad_out, void *stream);

/*
 * vqc_train_step -- one training evaluation: vqc_forward, vqc_loss_grad with
 * `loss_kind` and `target`, and vqc_backward with that cotangent, in one call
 * (Sec. 3 "Gate Application and Differentiation"; Sec. 4.2.3 objective).  On
 * the resident path this is a single launch: the final state stays on chip
 * between the forward and the adjoint sweep and is never written to HBM.
 *   expvals [batch, n] written; grad_out [batch, n] receives the cotangent
 *   when not NULL; dparams [batch, P] ([P] with shared_params) / dinputs
 *   [batch, F] written (either may be NULL); workspace:
 *   vqc_workspace_bytes(c, batch, 2) bytes, 256-byte aligned (on the resident
 *   path 0 bytes / NULL unless shared_params).
 * On the streaming path the batch halves run on two streams (see
 * vqc_workspace_bytes).  Results equal those of the three separate calls up
 * to float rounding: with the generated kernels the step builds the state
 * after every qubit's leading rotations (those before any entangler on it) as
 * a product state and takes their gradients from lambda contracted against
 * it, where the separate calls run them as gates (on the streaming path with
 * a plan of its own, which vqc_circuit_info reports).  Errors: those of the
 * three calls.
 */
int vqc_train_step(const vqc_circuit *c, int64_t batch, const float *params, const float *inputs,
                   int32_t loss_kind, const float *target, float *expvals, float *grad_out,
                   float *dparams, float *dinputs, void *workspace, size_t workspace_bytes,
                   void *stream);

/*
 * vqc_train_step_noalloc -- vqc_train_step for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  The workspace is a static device array of
 * VQC_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends; the call itself allocates and frees nothing.
 * Arguments, results and errors as vqc_train_step without the workspace, plus
 * VQC_ERR_TOO_LARGE when vqc_workspace_bytes(c, batch, 2) exceeds
 * VQC_NOALLOC_SCRATCH_BYTES (e.g. 16 qubits on the streaming path: about 1.5
 * MiB per sample).  Every call on one GPU uses that GPU's single array and
 * finds there what the last call left (the call clears what must start at
 * zero): calls that overlap on one GPU, from other streams or threads, race
 * and must be ordered by the caller.  The whole step runs on `stream` (no side
 * stream).
 */
#define VQC_NOALLOC_SCRATCH_BYTES 67108864
int vqc_train_step_noalloc(const vqc_circuit *c, int64_t batch, const float *params,
                           const float *inputs, int32_t loss_kind, const float *target,
                           float *expvals, float *grad_out, float *dparams, float *dinputs,
                           void *stream);

/*
 * vqc_fd_backward -- the same gradient as vqc_backward by central differences
 * (the matched central finite-difference training policy of Sec. 4.2.3 and
 * the "no autograd" ablation of Sec. 4.2.4; kept to compare the mechanisms):
 * for every sample, parameter and input s,
 *   d L / d s = sum_q g[b,q] (E_q(s + h) - E_q(s - h)) / (2 h),
 * from 2 (P + F) shifted forward evaluations per sample, run as one batch on
 * the resident path and, on the streaming path, as one batch per chunk of
 * slots (as many slots as keep the shifted copies' states within 2 GiB).
 * h > 0.  workspace: vqc_workspace_bytes(c, batch, 3) bytes (the shifted
 * copies' E rows, and their states when streaming), 256-byte aligned.
 * Outputs and shared_params as in vqc_backward.  Errors: VQC_ERR_INVALID_ARG,
 * VQC_ERR_TOO_LARGE, VQC_ERR_WORKSPACE, VQC_ERR_HIP.
 */
int vqc_fd_backward(const vqc_circuit *c, int64_t batch, const float *params, const float *inputs,
                    const float *grad_out, float h, void *workspace, size_t workspace_bytes,
                    float *dparams, float *dinputs, void *stream);

/* Introspection of a compiled circuit (host-side values only). */
typedef struct {
    int32_t n_qubits, n_params, n_inputs, n_ops;
    int32_t n_rotations;    /* primitive rotations (ROT counts 3) */
    int32_t path;           /* VQC_PATH_RESIDENT or VQC_PATH_STREAM */
    int32_t tile_qubits;    /* qubits held on chip by one workgroup */
    int32_t threads;        /* workgroup size */
    int32_t fwd_passes;     /* kernel passes of the forward (1 when resident) */
    int32_t bwd_passes;     /* kernel passes of the backward */
    int32_t fwd_exchanges;  /* on-chip layout exchanges in the forward */
    int32_t bwd_exchanges;  /* on-chip layout exchanges in the backward */
    int32_t fwd_instructions, bwd_instructions;
    int32_t lds_bytes_fwd, lds_bytes_bwd;
    int32_t engine;         /* VQC_ENGINE_* */
    int32_t shared_params;  /* the compile option */
    /* streaming path, generated kernels: rotations that vqc_train_step builds
       as a product state instead of running them (0: none), and that step's
       passes; 0 otherwise */
    int32_t step_head_rotations, step_fwd_passes, step_bwd_passes;
    int32_t reserved[3];
} vqc_info;
int vqc_circuit_info(const vqc_circuit *c, vqc_info *info);

/*
 * vqc_jit_check -- generate the run-time kernels of a compiled circuit (host-
 * only handles included) and compile them for gfx950 without loading them.
 * Needs no GPU.  Errors: VQC_ERR_INVALID_ARG (NULL), VQC_ERR_UNSUPPORTED (the
 * compiler rejected the source; vqc_last_error() holds its log).
 */
int vqc_jit_check(const vqc_circuit *c);

/* Message of the last failure on the calling thread ("" if none). */
const char *vqc_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* VQC_ABI_H_ */
