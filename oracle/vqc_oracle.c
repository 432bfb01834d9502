/*
 * vqc_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, double-precision CPU reference for the batched statevector
 * forward pass of a static parametrized circuit and for its exact
 * vector-Jacobian product.  Only the test suite, the package's smoke check and
 * the benchmark's CPU-baseline leg may load this library; the product path
 * (the HIP library and its Python binding) never does.  It shares no code,
 * header, table or helper with the HIP path.
 *
 * What it follows:
 *   - Sec. 3 "Compile-Once Lowering and Execution" and Algorithm 1 (execute
 *     phase): the state starts as |0...0> (or the caller's Psi_0, which
 *     Algorithm 1 accepts as an optional input), every gate of the fixed
 *     sequence is applied in order with its angles resolved from the current
 *     parameters.  Every gate is applied as its own full 2^k x 2^k matrix
 *     (k <= 3 qubits), written from the gate's definition -- no gate is
 *     decomposed into others.
 *   - Algorithm 1, return statement: E[:,j] = sum_k (-1)^{k_j} |Psi[:,k]|^2.
 *   - Sec. 3 "Gate Application and Differentiation": exact gradients of the
 *     trainable parameters.  Here they are obtained by the chain rule over
 *     *stored* intermediate states with explicit derivative matrices dU/dtheta
 *     (the memory-hungry scheme the paper attributes to autograd, Sec. 3
 *     "Complexity and Tradeoffs"), never by uncomputing states.
 *
 * Gate definitions (the OpenQASM standard gate library's matrices; the paper
 * names OpenQASM as its input format, Sec. 3):
 *   R_P(t) = exp(-i t P / 2) for P in {X, Y, Z};
 *   ROT(phi, theta, omega) = RZ(omega) RY(theta) RZ(phi);
 *   P(l) = diag(1, e^{il}); U3(t, p, l) = [[c, -e^{il} s], [e^{ip} s, e^{i(p+l)} c]]
 *     with c = cos t/2, s = sin t/2; U2(p, l) = U3(pi/2, p, l);
 *   H, S = diag(1, i), T = diag(1, e^{i pi/4}), SX = sqrt(X) = (1/2)[[1+i, 1-i], [1-i, 1+i]]
 *     and their inverses; controlled gates act on the target when the control is 1;
 *   R_PP(t) = exp(-i t P(x)P / 2) for PP in {XX, YY, ZZ}.
 * Angle slots are affine in one source: angle = mul * value + add, where value
 * is a parameter or an input of the sample, or angle = add for a constant.
 * Qubit j is bit j of the basis index; wire i of a gate is bit i of the gate
 * matrix's index (for a controlled gate wire 0 is the control).
 *
 * Everything is complex128; angles arrive as doubles (the float32 inputs of
 * the GPU path upcast by the caller).
 */
#include <complex.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef double complex cplx;

static const double ORC_PI = 3.14159265358979323846;

enum {
    ORC_RX = 0, ORC_RY, ORC_RZ, ORC_ROT, ORC_CNOT, ORC_CZ,
    ORC_ID, ORC_X, ORC_Y, ORC_Z, ORC_H, ORC_S, ORC_SDG, ORC_T, ORC_TDG, ORC_SX, ORC_SXDG,
    ORC_P, ORC_U2, ORC_U3,
    ORC_CY, ORC_CH, ORC_SWAP, ORC_CRX, ORC_CRY, ORC_CRZ, ORC_CP, ORC_RXX, ORC_RYY, ORC_RZZ,
    ORC_CCX, ORC_CSWAP,
    ORC_NKIND
};
enum { ORC_PARAM = 0, ORC_INPUT = 1, ORC_CONST = 2 };

/* One gate.  88 bytes; the Python wrapper builds the matching record. */
typedef struct {
    int32_t kind;
    int32_t w[3];        /* wires; unused ones are -1 */
    int32_t src[3];      /* angle source per slot */
    int32_t idx[3];      /* param / input index per slot */
    double mul[3];       /* angle = mul * value + add (param / input) */
    double add[3];       /* angle = add (constant) */
} oracle_op;

static int arity(int kind) {
    switch (kind) {
    case ORC_CNOT: case ORC_CZ: case ORC_CY: case ORC_CH: case ORC_SWAP: case ORC_CRX:
    case ORC_CRY: case ORC_CRZ: case ORC_CP: case ORC_RXX: case ORC_RYY: case ORC_RZZ:
        return 2;
    case ORC_CCX: case ORC_CSWAP: return 3;
    default: return 1;
    }
}

static int n_angles(int kind) {
    switch (kind) {
    case ORC_RX: case ORC_RY: case ORC_RZ: case ORC_P: case ORC_CRX: case ORC_CRY:
    case ORC_CRZ: case ORC_CP: case ORC_RXX: case ORC_RYY: case ORC_RZZ:
        return 1;
    case ORC_U2: return 2;
    case ORC_ROT: case ORC_U3: return 3;
    default: return 0;
    }
}

/* ---- 2x2 building blocks ------------------------------------------------ */
typedef struct { cplx m[2][2]; } mat2;

static mat2 mk2(cplx a, cplx b, cplx c, cplx d) {
    mat2 u = {{{a, b}, {c, d}}};
    return u;
}
/* R_P(t) = exp(-i t P/2) written out, and d/dt of it */
static mat2 m_rx(double t) { double c = cos(t / 2), s = sin(t / 2); return mk2(c, -I * s, -I * s, c); }
static mat2 m_ry(double t) { double c = cos(t / 2), s = sin(t / 2); return mk2(c, -s, s, c); }
static mat2 m_rz(double t) { return mk2(cexp(-I * t / 2), 0, 0, cexp(I * t / 2)); }
static mat2 d_rx(double t) {
    double c = cos(t / 2), s = sin(t / 2);
    return mk2(-0.5 * s, -0.5 * I * c, -0.5 * I * c, -0.5 * s);
}
static mat2 d_ry(double t) {
    double c = cos(t / 2), s = sin(t / 2);
    return mk2(-0.5 * s, -0.5 * c, 0.5 * c, -0.5 * s);
}
static mat2 d_rz(double t) { return mk2(-0.5 * I * cexp(-I * t / 2), 0, 0, 0.5 * I * cexp(I * t / 2)); }
static mat2 mul2(mat2 a, mat2 b) {
    mat2 r;
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j)
            r.m[i][j] = a.m[i][0] * b.m[0][j] + a.m[i][1] * b.m[1][j];
    return r;
}

/* U3(t, p, l) and its partial derivative w.r.t. argument d (0: t, 1: p, 2: l) */
static mat2 m_u3(double t, double p, double l, int d) {
    double c = cos(t / 2), s = sin(t / 2);
    cplx ep = cexp(I * p), el = cexp(I * l), epl = cexp(I * (p + l));
    switch (d) {
    case 0: return mk2(-0.5 * s, -0.5 * el * c, 0.5 * ep * c, -0.5 * epl * s);
    case 1: return mk2(0, 0, I * ep * s, I * epl * c);
    case 2: return mk2(0, -I * el * s, 0, I * epl * c);
    default: return mk2(c, -el * s, ep * s, epl * c);
    }
}

/* The 2x2 matrix of a one-qubit gate (d < 0) or its derivative w.r.t. slot d. */
static mat2 one_qubit(int kind, const double *a, int d) {
    const double r2 = 1.0 / sqrt(2.0);
    switch (kind) {
    case ORC_RX: return d < 0 ? m_rx(a[0]) : d_rx(a[0]);
    case ORC_RY: return d < 0 ? m_ry(a[0]) : d_ry(a[0]);
    case ORC_RZ: return d < 0 ? m_rz(a[0]) : d_rz(a[0]);
    case ORC_ROT: {
        mat2 x = (d == 2) ? d_rz(a[2]) : m_rz(a[2]);
        mat2 y = (d == 1) ? d_ry(a[1]) : m_ry(a[1]);
        mat2 z = (d == 0) ? d_rz(a[0]) : m_rz(a[0]);
        return mul2(x, mul2(y, z));
    }
    case ORC_ID: return mk2(1, 0, 0, 1);
    case ORC_X: return mk2(0, 1, 1, 0);
    case ORC_Y: return mk2(0, -I, I, 0);
    case ORC_Z: return mk2(1, 0, 0, -1);
    case ORC_H: return mk2(r2, r2, r2, -r2);
    case ORC_S: return mk2(1, 0, 0, I);
    case ORC_SDG: return mk2(1, 0, 0, -I);
    case ORC_T: return mk2(1, 0, 0, cexp(I * ORC_PI / 4));
    case ORC_TDG: return mk2(1, 0, 0, cexp(-I * ORC_PI / 4));
    case ORC_SX: return mk2(0.5 * (1 + I), 0.5 * (1 - I), 0.5 * (1 - I), 0.5 * (1 + I));
    case ORC_SXDG: return mk2(0.5 * (1 - I), 0.5 * (1 + I), 0.5 * (1 + I), 0.5 * (1 - I));
    case ORC_P: return d < 0 ? mk2(1, 0, 0, cexp(I * a[0])) : mk2(0, 0, 0, I * cexp(I * a[0]));
    case ORC_U2: return m_u3(ORC_PI / 2, a[0], a[1], d < 0 ? -1 : d + 1);
    case ORC_U3: return m_u3(a[0], a[1], a[2], d);
    default: return mk2(0, 0, 0, 0);
    }
}

/* the target's 2x2 block of a controlled gate */
static mat2 controlled_block(int kind, const double *a, int d) {
    switch (kind) {
    case ORC_CNOT: return one_qubit(ORC_X, a, -1);
    case ORC_CZ: return one_qubit(ORC_Z, a, -1);
    case ORC_CY: return one_qubit(ORC_Y, a, -1);
    case ORC_CH: return one_qubit(ORC_H, a, -1);
    case ORC_CRX: return one_qubit(ORC_RX, a, d);
    case ORC_CRY: return one_qubit(ORC_RY, a, d);
    case ORC_CRZ: return one_qubit(ORC_RZ, a, d);
    default: return one_qubit(ORC_P, a, d); /* ORC_CP */
    }
}

/*
 * The 2^k x 2^k matrix (row-major, k = arity) of a gate, or (d >= 0) its
 * derivative w.r.t. angle slot d.  Index bit i of the matrix is wire i.
 */
static void gate_matrix(int kind, const double *a, int d, cplx *M) {
    const int k = arity(kind), dim = 1 << k;
    memset(M, 0, sizeof(cplx) * dim * dim);
    if (k == 1) {
        mat2 u = one_qubit(kind, a, d);
        for (int i = 0; i < 2; ++i)
            for (int j = 0; j < 2; ++j) M[i * 2 + j] = u.m[i][j];
        return;
    }
    switch (kind) {
    case ORC_CNOT: case ORC_CZ: case ORC_CY: case ORC_CH: case ORC_CRX: case ORC_CRY:
    case ORC_CRZ: case ORC_CP: {
        /* |0><0|_c (x) I + |1><1|_c (x) U; the derivative has no |0> block */
        mat2 u = controlled_block(kind, a, d);
        if (d < 0) { M[0 * 4 + 0] = 1; M[2 * 4 + 2] = 1; }
        for (int i = 0; i < 2; ++i)
            for (int j = 0; j < 2; ++j) M[(1 + 2 * i) * 4 + (1 + 2 * j)] = u.m[i][j];
        return;
    }
    case ORC_SWAP:
        for (int l = 0; l < 4; ++l) M[(((l & 1) << 1) | (l >> 1)) * 4 + l] = 1;
        return;
    case ORC_RXX: case ORC_RYY: case ORC_RZZ: {
        /* cos(t/2) I - i sin(t/2) G, G = P (x) P */
        double c = cos(a[0] / 2), s = sin(a[0] / 2);
        cplx ci = d < 0 ? c : -0.5 * s;       /* coefficient of I */
        cplx cg = d < 0 ? -I * s : -0.5 * I * c; /* coefficient of G */
        for (int l = 0; l < 4; ++l) {
            M[l * 4 + l] += ci;
            int par = (l & 1) ^ (l >> 1);
            if (kind == ORC_RZZ) M[l * 4 + l] += cg * (par ? -1.0 : 1.0);
            else if (kind == ORC_RXX) M[(l ^ 3) * 4 + l] += cg;
            else M[(l ^ 3) * 4 + l] += cg * (par ? 1.0 : -1.0); /* YY|ab> = -(-1)^{a+b}|~a~b> */
        }
        return;
    }
    case ORC_CCX:
        for (int l = 0; l < 8; ++l) M[((l & 3) == 3 ? l ^ 4 : l) * 8 + l] = 1;
        return;
    case ORC_CSWAP:
        for (int l = 0; l < 8; ++l) {
            int r = l;
            if (l & 1) r = (l & 1) | (((l >> 2) & 1) << 1) | (((l >> 1) & 1) << 2);
            M[r * 8 + l] = 1;
        }
        return;
    default:
        return;
    }
}

/* psi <- M psi on wires w[0..k) (M any 2^k x 2^k matrix, row-major) */
static void apply_k(cplx *psi, int n, const int32_t *w, int k, const cplx *M) {
    const size_t N = (size_t)1 << n;
    const int dim = 1 << k;
    size_t mask = 0, off[8];
    for (int i = 0; i < k; ++i) mask |= (size_t)1 << w[i];
    for (int l = 0; l < dim; ++l) {
        off[l] = 0;
        for (int i = 0; i < k; ++i)
            if ((l >> i) & 1) off[l] |= (size_t)1 << w[i];
    }
    cplx in[8];
    for (size_t x = 0; x < N; ++x) {
        if (x & mask) continue;
        for (int l = 0; l < dim; ++l) in[l] = psi[x | off[l]];
        for (int r = 0; r < dim; ++r) {
            cplx acc = 0;
            for (int l = 0; l < dim; ++l) acc += M[r * dim + l] * in[l];
            psi[x | off[r]] = acc;
        }
    }
}

static void resolve_angles(const oracle_op *op, int b, const double *params, int P,
                           const double *inputs, int F, double *ang) {
    for (int s = 0; s < n_angles(op->kind); ++s) {
        if (op->src[s] == ORC_PARAM)
            ang[s] = op->mul[s] * params[(size_t)b * P + op->idx[s]] + op->add[s];
        else if (op->src[s] == ORC_INPUT)
            ang[s] = op->mul[s] * inputs[(size_t)b * F + op->idx[s]] + op->add[s];
        else
            ang[s] = op->add[s];
    }
}

/* psi <- U psi, or U^dagger psi (adjoint) */
static void apply_op(cplx *psi, int n, const oracle_op *op, const double *ang, int adjoint) {
    const int k = arity(op->kind), dim = 1 << k;
    cplx M[64], A[64];
    gate_matrix(op->kind, ang, -1, M);
    if (adjoint) {
        for (int r = 0; r < dim; ++r)
            for (int c = 0; c < dim; ++c) A[r * dim + c] = conj(M[c * dim + r]);
        apply_k(psi, n, op->w, k, A);
    } else {
        apply_k(psi, n, op->w, k, M);
    }
}

/* E[j] = sum_x (-1)^{x_j} |psi[x]|^2  (Algorithm 1, return statement) */
static void z_expectations(const cplx *psi, int n, double *e) {
    size_t N = (size_t)1 << n;
    for (int j = 0; j < n; ++j) {
        double acc = 0.0;
        for (size_t x = 0; x < N; ++x) {
            double p = creal(psi[x]) * creal(psi[x]) + cimag(psi[x]) * cimag(psi[x]);
            acc += ((x >> j) & 1) ? -p : p;
        }
        e[j] = acc;
    }
}

static int validate(const oracle_op *ops, int n_ops, int n, int P, int F) {
    if (n < 1 || n > 24 || n_ops < 0) return -1;
    for (int k = 0; k < n_ops; ++k) {
        const oracle_op *o = &ops[k];
        if (o->kind < 0 || o->kind >= ORC_NKIND) return -1;
        for (int i = 0; i < arity(o->kind); ++i) {
            if (o->w[i] < 0 || o->w[i] >= n) return -1;
            for (int j = 0; j < i; ++j)
                if (o->w[j] == o->w[i]) return -1;
        }
        for (int s = 0; s < n_angles(o->kind); ++s) {
            if (o->src[s] == ORC_PARAM && (o->idx[s] < 0 || o->idx[s] >= P)) return -1;
            if (o->src[s] == ORC_INPUT && (o->idx[s] < 0 || o->idx[s] >= F)) return -1;
            if (o->src[s] < ORC_PARAM || o->src[s] > ORC_CONST) return -1;
        }
    }
    return 0;
}

static void set_threads(int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/*
 * Forward pass for B samples.  expvals: [B, n].  states (optional): [B, 2^n]
 * complex128 final states.  psi0: NULL for |0...0>, else [B][2^n] complex128
 * initial states.  If shift_op >= 0, angle slot shift_slot of gate shift_op
 * is offset by `delta` (after the affine map) in every sample (used by the
 * shift-rule and finite-difference checks of the tests).  Returns 0, or -1 on
 * invalid input, -2 on allocation failure.
 */
int oracle_forward(const oracle_op *ops, int n_ops, int n, int B,
                   const double *params, int P, const double *inputs, int F,
                   double *expvals, double *states,
                   int shift_op, int shift_slot, double delta, int nthreads,
                   const double *psi0) {
    if (validate(ops, n_ops, n, P, F) != 0 || B < 0) return -1;
    set_threads(nthreads);
    size_t N = (size_t)1 << n;
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        cplx *psi = (cplx *)calloc(N, sizeof(cplx));
        if (!psi) { err = -2; continue; }
        if (psi0) memcpy(psi, psi0 + (size_t)b * N * 2, N * sizeof(cplx));
        else psi[0] = 1.0;
        for (int k = 0; k < n_ops; ++k) {
            double ang[3] = {0, 0, 0};
            resolve_angles(&ops[k], b, params, P, inputs, F, ang);
            if (k == shift_op) ang[shift_slot] += delta;
            apply_op(psi, n, &ops[k], ang, 0);
        }
        z_expectations(psi, n, expvals + (size_t)b * n);
        if (states) memcpy(states + (size_t)b * N * 2, psi, N * sizeof(cplx));
        free(psi);
    }
    return err;
}

/*
 * Vector-Jacobian product.  With cotangent g = grad_out[b, :] the scalar is
 * L_b = sum_j g_j E[b, j] = <psi_G| H |psi_G>, H = sum_j g_j Z_j.  For gate k
 * and angle t of that gate,
 *     dL_b/dt = 2 Re < lam_k | (dU_k/dt) | psi_{k-1} >,
 *     lam_G = H psi_G,  lam_{k-1} = U_k^dagger lam_k,
 * with every psi_k taken from the stored forward states.  By the chain rule a
 * slot t = mul * value + add contributes mul * dL_b/dt to the parameter /
 * input it reads (constant angles contribute nothing).  dparams [B, P] and
 * dinputs [B, F] are overwritten; expvals [B, n] (optional) receives E.
 */
int oracle_vjp(const oracle_op *ops, int n_ops, int n, int B,
               const double *params, int P, const double *inputs, int F,
               const double *grad_out, double *dparams, double *dinputs,
               double *expvals, int nthreads, const double *psi0) {
    if (validate(ops, n_ops, n, P, F) != 0 || B < 0) return -1;
    set_threads(nthreads);
    size_t N = (size_t)1 << n;
    int err = 0;
    memset(dparams, 0, sizeof(double) * (size_t)B * (size_t)P);
    memset(dinputs, 0, sizeof(double) * (size_t)B * (size_t)F);
#pragma omp parallel for schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        cplx *st = (cplx *)malloc(sizeof(cplx) * N * ((size_t)n_ops + 1));
        cplx *lam = (cplx *)malloc(sizeof(cplx) * N);
        cplx *tmp = (cplx *)malloc(sizeof(cplx) * N);
        if (!st || !lam || !tmp) { free(st); free(lam); free(tmp); err = -2; continue; }
        /* forward, keeping psi_0 .. psi_G */
        if (psi0) {
            memcpy(st, psi0 + (size_t)b * N * 2, sizeof(cplx) * N);
        } else {
            memset(st, 0, sizeof(cplx) * N);
            st[0] = 1.0;
        }
        for (int k = 0; k < n_ops; ++k) {
            double ang[3] = {0, 0, 0};
            resolve_angles(&ops[k], b, params, P, inputs, F, ang);
            memcpy(st + (size_t)(k + 1) * N, st + (size_t)k * N, sizeof(cplx) * N);
            apply_op(st + (size_t)(k + 1) * N, n, &ops[k], ang, 0);
        }
        const cplx *psiG = st + (size_t)n_ops * N;
        if (expvals) z_expectations(psiG, n, expvals + (size_t)b * n);
        /* lam_G = H psi_G */
        const double *g = grad_out + (size_t)b * n;
        for (size_t x = 0; x < N; ++x) {
            double h = 0.0;
            for (int j = 0; j < n; ++j) h += ((x >> j) & 1) ? -g[j] : g[j];
            lam[x] = h * psiG[x];
        }
        for (int k = n_ops - 1; k >= 0; --k) {
            const oracle_op *op = &ops[k];
            double ang[3] = {0, 0, 0};
            resolve_angles(op, b, params, P, inputs, F, ang);
            const cplx *prev = st + (size_t)k * N; /* psi_{k-1} in 1-based terms */
            for (int s = 0; s < n_angles(op->kind); ++s) {
                if (op->src[s] == ORC_CONST) continue;
                cplx D[64];
                gate_matrix(op->kind, ang, s, D);
                memcpy(tmp, prev, sizeof(cplx) * N);
                apply_k(tmp, n, op->w, arity(op->kind), D);
                double acc = 0.0;
                for (size_t x = 0; x < N; ++x) acc += creal(conj(lam[x]) * tmp[x]);
                acc *= 2.0 * op->mul[s];
                if (op->src[s] == ORC_PARAM) dparams[(size_t)b * P + op->idx[s]] += acc;
                else dinputs[(size_t)b * F + op->idx[s]] += acc;
            }
            apply_op(lam, n, op, ang, 1);
        }
        free(st); free(lam); free(tmp);
    }
    return err;
}

/* Size of the record above, so the wrapper can check its own layout. */
int oracle_op_size(void) { return (int)sizeof(oracle_op); }
