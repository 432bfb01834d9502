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
 *     sequence is applied in order with its angle resolved from the current
 *     parameters.
 *   - Algorithm 1, return statement: E[:,j] = sum_k (-1)^{k_j} |Psi[:,k]|^2.
 *   - Sec. 3 "Gate Application and Differentiation": exact gradients of the
 *     trainable parameters.  Here they are obtained by the chain rule over
 *     *stored* intermediate states with explicit derivative matrices dU/dtheta
 *     (the memory-hungry scheme the paper attributes to autograd, Sec. 3
 *     "Complexity and Tradeoffs"), never by uncomputing states.
 *
 * Readings (the paper does not fix them): R_P(t) = exp(-i t P / 2) for
 * P in {X, Y, Z}; ROT(phi, theta, omega) = RZ(omega) RY(theta) RZ(phi);
 * qubit j is bit j of the basis index.
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

enum { ORC_RX = 0, ORC_RY = 1, ORC_RZ = 2, ORC_ROT = 3, ORC_CNOT = 4, ORC_CZ = 5 };
enum { ORC_PARAM = 0, ORC_INPUT = 1, ORC_CONST = 2 };

/* One gate.  64 bytes; the Python wrapper builds the matching record. */
typedef struct {
    int32_t kind;
    int32_t w0, w1;      /* target (1q) | control,target (CNOT) | a,b (CZ) */
    int32_t src[3];      /* angle source per slot */
    int32_t idx[3];      /* param / input index per slot */
    int32_t pad;
    double val[3];       /* constant angle per slot */
} oracle_op;

typedef struct { cplx m[2][2]; } mat2;

static int n_angles(int kind) {
    switch (kind) {
    case ORC_RX: case ORC_RY: case ORC_RZ: return 1;
    case ORC_ROT: return 3;
    default: return 0;
    }
}

/* ---- single-qubit matrices, R_P(t) = exp(-i t P/2) written out ---------- */
static mat2 m_rx(double t) {
    double c = cos(t / 2), s = sin(t / 2);
    mat2 u = {{{c, -I * s}, {-I * s, c}}};
    return u;
}
static mat2 m_ry(double t) {
    double c = cos(t / 2), s = sin(t / 2);
    mat2 u = {{{c, -s}, {s, c}}};
    return u;
}
static mat2 m_rz(double t) {
    mat2 u = {{{cexp(-I * t / 2), 0}, {0, cexp(I * t / 2)}}};
    return u;
}
/* derivatives d/dt of the three matrices above */
static mat2 d_rx(double t) {
    double c = cos(t / 2), s = sin(t / 2);
    mat2 u = {{{-0.5 * s, -0.5 * I * c}, {-0.5 * I * c, -0.5 * s}}};
    return u;
}
static mat2 d_ry(double t) {
    double c = cos(t / 2), s = sin(t / 2);
    mat2 u = {{{-0.5 * s, -0.5 * c}, {0.5 * c, -0.5 * s}}};
    return u;
}
static mat2 d_rz(double t) {
    mat2 u = {{{-0.5 * I * cexp(-I * t / 2), 0}, {0, 0.5 * I * cexp(I * t / 2)}}};
    return u;
}
static mat2 mul2(mat2 a, mat2 b) {
    mat2 r;
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j)
            r.m[i][j] = a.m[i][0] * b.m[0][j] + a.m[i][1] * b.m[1][j];
    return r;
}
static mat2 dagger2(mat2 a) {
    mat2 r;
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 2; ++j)
            r.m[i][j] = conj(a.m[j][i]);
    return r;
}

/* The matrix of a one-qubit gate, or its derivative w.r.t. angle slot `d`
 * (d < 0: the matrix itself).  ROT is the explicit product
 * RZ(omega) RY(theta) RZ(phi) and its three partial derivatives. */
static mat2 gate_matrix(int kind, const double *ang, int d) {
    switch (kind) {
    case ORC_RX: return d < 0 ? m_rx(ang[0]) : d_rx(ang[0]);
    case ORC_RY: return d < 0 ? m_ry(ang[0]) : d_ry(ang[0]);
    case ORC_RZ: return d < 0 ? m_rz(ang[0]) : d_rz(ang[0]);
    default: {
        mat2 a = (d == 2) ? d_rz(ang[2]) : m_rz(ang[2]);
        mat2 b = (d == 1) ? d_ry(ang[1]) : m_ry(ang[1]);
        mat2 c = (d == 0) ? d_rz(ang[0]) : m_rz(ang[0]);
        return mul2(a, mul2(b, c));
    }
    }
}

/* psi <- U on qubit q (any 2x2, unitary or not) */
static void apply_1q(cplx *psi, int n, int q, mat2 u) {
    size_t N = (size_t)1 << n, bit = (size_t)1 << q;
    for (size_t x = 0; x < N; ++x) {
        if (x & bit) continue;
        cplx a0 = psi[x], a1 = psi[x | bit];
        psi[x] = u.m[0][0] * a0 + u.m[0][1] * a1;
        psi[x | bit] = u.m[1][0] * a0 + u.m[1][1] * a1;
    }
}

/* CNOT(c, t): |x> -> |x xor (x_c << t)> ; self-inverse */
static void apply_cnot(cplx *psi, int n, int c, int t) {
    size_t N = (size_t)1 << n, bc = (size_t)1 << c, bt = (size_t)1 << t;
    for (size_t x = 0; x < N; ++x) {
        if ((x & bc) && !(x & bt)) {
            cplx tmp = psi[x];
            psi[x] = psi[x | bt];
            psi[x | bt] = tmp;
        }
    }
}

/* CZ(a, b): |x> -> (-1)^{x_a x_b} |x> ; self-inverse */
static void apply_cz(cplx *psi, int n, int a, int b) {
    size_t N = (size_t)1 << n, ba = (size_t)1 << a, bb = (size_t)1 << b;
    for (size_t x = 0; x < N; ++x)
        if ((x & ba) && (x & bb)) psi[x] = -psi[x];
}

static void resolve_angles(const oracle_op *op, int b, const double *params, int P,
                           const double *inputs, int F, double *ang) {
    for (int s = 0; s < n_angles(op->kind); ++s) {
        if (op->src[s] == ORC_PARAM) ang[s] = params[(size_t)b * P + op->idx[s]];
        else if (op->src[s] == ORC_INPUT) ang[s] = inputs[(size_t)b * F + op->idx[s]];
        else ang[s] = op->val[s];
    }
}

static void apply_op(cplx *psi, int n, const oracle_op *op, const double *ang, int adjoint) {
    if (op->kind == ORC_CNOT) { apply_cnot(psi, n, op->w0, op->w1); return; }
    if (op->kind == ORC_CZ) { apply_cz(psi, n, op->w0, op->w1); return; }
    mat2 u = gate_matrix(op->kind, ang, -1);
    apply_1q(psi, n, op->w0, adjoint ? dagger2(u) : u);
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
        if (o->kind < ORC_RX || o->kind > ORC_CZ) return -1;
        if (o->w0 < 0 || o->w0 >= n) return -1;
        if (o->kind >= ORC_CNOT && (o->w1 < 0 || o->w1 >= n || o->w1 == o->w0)) return -1;
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
 * complex128 final states.  If shift_op >= 0, angle slot shift_slot of gate
 * shift_op is offset by `delta` in every sample (used by the parameter-shift
 * and finite-difference checks of the tests).  Returns 0, or -1 on invalid
 * input, -2 on allocation failure.
 */
/* psi0: NULL for |0...0>, else [B][2^n] complex128 initial states. */
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
 * with every psi_k taken from the stored forward states.  Contributions are
 * summed into the parameter / input slot the angle reads from (constant
 * angles get none).  dparams [B, P] and dinputs [B, F] are overwritten;
 * expvals [B, n] (optional) receives E.
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
                memcpy(tmp, prev, sizeof(cplx) * N);
                apply_1q(tmp, n, op->w0, gate_matrix(op->kind, ang, s));
                double acc = 0.0;
                for (size_t x = 0; x < N; ++x) acc += creal(conj(lam[x]) * tmp[x]);
                acc *= 2.0;
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
