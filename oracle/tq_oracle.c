/*
 * tq_oracle.c -- the oracle: a plain, slow, complex128 CPU state-vector
 * simulator of batched parameterized circuits.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this library.  The product path
 * (the HIP library) never links, calls or includes anything from here, and
 * this file shares no code with it: it has its own blob parser, its own gate
 * table and its own sampler.
 *
 * What it computes (TensorFlow Quantum, arXiv:2003.02989):
 *  - the final state of each circuit of the batch, psi_b = W_G ... W_1 |0..0>,
 *    with every parameter resolved from the symbol values (Sec. "Cirq",
 *    ParamResolver semantics; Sec. "Quantum Neural Networks",
 *    eqs. full_par_circ, layer_blocks, Pauli_decomp); the gates include the
 *    exponential exp(-i eta P) of a Pauli string of any weight, applied as
 *    cos(eta) psi - i sin(eta) P psi (eq. cs_decomp);
 *  - expectation values <psi_b| h_{b,k} |psi_b> of Pauli sums
 *    h = sum_t c_t P_t (Sec. "Sampling and Expectations",
 *    eqs. cost_lincomb and qee_lincomb);
 *  - adjoint-method gradients of sum_k g_{b,k} <h_{b,k}> with respect to the
 *    symbol values (Sec. "Adjoint Gradient Backpropagation in Simulations";
 *    the effective Hamiltonian H_g of Sec. "Autodifferentiation through
 *    hybrid quantum-classical backpropagation"; shared symbols add up over
 *    their occurrences by the chain rule, eq. chain_rule);
 *  - noisy circuits by trajectories (Sec. "Noise in qsim"): each row draws
 *    one Pauli per channel from a counter stream and is then a pure circuit;
 *  - expectations estimated from a finite number of measurement shots per
 *    term (SampledExpectation);
 *  - gradients by the parameter-shift rule (exact or from sampled
 *    expectations) and by central finite differences (Sec. "Parameter shift
 *    methods", Sec. "Finite difference methods");
 *  - bitstring samples drawn from |psi_i|^2 (Sec. "Sampling and Expectation
 *    Values") with the integer fixed-point rule and the SplitMix64 counter
 *    stream stated at the sampler below (the paper leaves both open).
 *
 * Every step is done gate by gate, on the full 2^n vector, with no fusion,
 * blocking or reordering.  Qubit q of an n-qubit circuit is bit (n-1-q) of an
 * amplitude index (qubit 0 is the most significant bit); a two-qubit gate on
 * (a, b) uses the local index 2*bit(a) + bit(b).
 *
 * Parity pins: see tests/test_oracle_*.py (closed forms printed in the paper,
 * gate identities, brute-force dense unitaries, parameter-shift and finite
 * differences).  No function here is "parity unpinned".
 */
#include <complex.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef double _Complex cplx;

/* ---------------------------------------------------------------- errors */
static __thread char g_err[512];
static int fail(const char *msg)
{
    snprintf(g_err, sizeof g_err, "%s", msg);
    return 1;
}
const char *orc_last_error(void) { return g_err; }

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------- op table */
enum {
    OP_H = 1, OP_X, OP_Y, OP_Z, OP_RX, OP_RY, OP_RZ, OP_XPOW, OP_YPOW, OP_ZPOW,
    OP_CZ, OP_CNOT, OP_CZPOW, OP_CNOTPOW, OP_XXPOW, OP_YYPOW, OP_ZZPOW, OP_RZZ,
    OP_SQRTX, OP_SQRTY, OP_SQRTW, OP_FSIM, OP_MATRIX1, OP_MATRIX2, OP_SWAP,
    OP_LAST = OP_SWAP,
    /* exp(-i eta P) of a Pauli string P of any weight (variable qubit count) */
    OP_PAULIEXP = 26,
    /* Pauli channel on one qubit: X, Y, Z with probabilities p_x, p_y, p_z
     * (three constant parameters), one Kraus operator drawn per trajectory */
    OP_PCHAN = 27
};

/* qubit count and parameter count of every opcode */
static int op_arity(int op, int *nq, int *np)
{
    switch (op) {
    case OP_H: case OP_X: case OP_Y: case OP_Z:
    case OP_SQRTX: case OP_SQRTY: case OP_SQRTW: case OP_MATRIX1:
        *nq = 1; *np = 0; return 0;
    case OP_RX: case OP_RY: case OP_RZ: case OP_XPOW: case OP_YPOW: case OP_ZPOW:
        *nq = 1; *np = 1; return 0;
    case OP_CZ: case OP_CNOT: case OP_MATRIX2: case OP_SWAP:
        *nq = 2; *np = 0; return 0;
    case OP_CZPOW: case OP_CNOTPOW: case OP_XXPOW: case OP_YYPOW: case OP_ZZPOW: case OP_RZZ:
        *nq = 2; *np = 1; return 0;
    case OP_FSIM:
        *nq = 2; *np = 2; return 0;
    case OP_PCHAN:
        *nq = 1; *np = 3; return 0;
    default:
        return 1;
    }
}

/* ----------------------------------------------------- small matrix math */
static void mat_eye(int d, cplx *m)
{
    for (int i = 0; i < d * d; i++) m[i] = 0;
    for (int i = 0; i < d; i++) m[i * d + i] = 1;
}
static void mat_mul(int d, const cplx *a, const cplx *b, cplx *out)
{
    cplx t[16];
    for (int i = 0; i < d; i++)
        for (int j = 0; j < d; j++) {
            cplx s = 0;
            for (int k = 0; k < d; k++) s += a[i * d + k] * b[k * d + j];
            t[i * d + j] = s;
        }
    memcpy(out, t, sizeof(cplx) * d * d);
}
static void kron2(const cplx *a, const cplx *b, cplx *out) /* 2x2 (x) 2x2 -> 4x4 */
{
    for (int i = 0; i < 2; i++)
        for (int j = 0; j < 2; j++)
            for (int k = 0; k < 2; k++)
                for (int l = 0; l < 2; l++)
                    out[(2 * i + k) * 4 + (2 * j + l)] = a[i * 2 + j] * b[k * 2 + l];
}

static const double SQRT1_2 = 0.70710678118654752440;

static void pauli2(int which, cplx *m) /* 0=I, 1=X, 2=Y, 3=Z */
{
    m[0] = m[1] = m[2] = m[3] = 0;
    switch (which) {
    case 0: m[0] = 1; m[3] = 1; break;
    case 1: m[1] = 1; m[2] = 1; break;
    case 2: m[1] = -I; m[2] = I; break;
    case 3: m[0] = 1; m[3] = -1; break;
    }
}

/* Involutory G raised to the power t, in the phase convention
 * G^t = exp(i*pi*t/2) * (cos(pi*t/2) I - i sin(pi*t/2) G). */
static void pow_involutory(int d, const cplx *g, double t, cplx *out)
{
    cplx ph = cexp(I * M_PI * t / 2.0);
    double c = cos(M_PI * t / 2.0), s = sin(M_PI * t / 2.0);
    for (int i = 0; i < d; i++)
        for (int j = 0; j < d; j++)
            out[i * d + j] = ph * ((i == j ? c : 0.0) - I * s * g[i * d + j]);
}
/* exp(-i*theta/2 * G) for involutory G */
static void rot_involutory(int d, const cplx *g, double theta, cplx *out)
{
    double c = cos(theta / 2.0), s = sin(theta / 2.0);
    for (int i = 0; i < d; i++)
        for (int j = 0; j < d; j++)
            out[i * d + j] = (i == j ? c : 0.0) - I * s * g[i * d + j];
}

/* The generator G (the involution) behind every pow / rotation opcode. */
static int op_generator(int op, cplx *g, int *d)
{
    cplx a[4], b[4];
    switch (op) {
    case OP_RX: case OP_XPOW: case OP_SQRTX: pauli2(1, g); *d = 2; return 0;
    case OP_RY: case OP_YPOW: case OP_SQRTY: pauli2(2, g); *d = 2; return 0;
    case OP_RZ: case OP_ZPOW: pauli2(3, g); *d = 2; return 0;
    case OP_SQRTW: { /* W = (X + Y) / sqrt(2) */
        pauli2(1, a); pauli2(2, b);
        for (int i = 0; i < 4; i++) g[i] = (a[i] + b[i]) * SQRT1_2;
        *d = 2; return 0; }
    case OP_CZ: case OP_CZPOW:
        mat_eye(4, g); g[15] = -1; *d = 4; return 0;
    case OP_CNOT: case OP_CNOTPOW:
        mat_eye(4, g); g[10] = 0; g[15] = 0; g[11] = 1; g[14] = 1; *d = 4; return 0;
    case OP_XXPOW: pauli2(1, a); kron2(a, a, g); *d = 4; return 0;
    case OP_YYPOW: pauli2(2, a); kron2(a, a, g); *d = 4; return 0;
    case OP_ZZPOW: case OP_RZZ: pauli2(3, a); kron2(a, a, g); *d = 4; return 0;
    default: return 1;
    }
}

/* Gate matrix of opcode `op` with resolved parameters `p` (radians for the
 * rotations, exponents for the pow gates, (theta, phi) for FSim).  `explicit`
 * holds the entries (re, im interleaved, row major) of MATRIX1 / MATRIX2. */
static int gate_matrix(int op, const double *p, const double *explicit_m, cplx *m, int *d)
{
    cplx g[16];
    switch (op) {
    case OP_H:
        *d = 2; m[0] = SQRT1_2; m[1] = SQRT1_2; m[2] = SQRT1_2; m[3] = -SQRT1_2; return 0;
    case OP_X: pauli2(1, m); *d = 2; return 0;
    case OP_Y: pauli2(2, m); *d = 2; return 0;
    case OP_Z: pauli2(3, m); *d = 2; return 0;
    case OP_CZ: case OP_CNOT:
        return op_generator(op, m, d);
    case OP_SWAP:
        mat_eye(4, m); m[5] = 0; m[10] = 0; m[6] = 1; m[9] = 1; *d = 4; return 0;
    case OP_RX: case OP_RY: case OP_RZ: case OP_RZZ:
        op_generator(op, g, d); rot_involutory(*d, g, p[0], m); return 0;
    case OP_XPOW: case OP_YPOW: case OP_ZPOW: case OP_CZPOW: case OP_CNOTPOW:
    case OP_XXPOW: case OP_YYPOW: case OP_ZZPOW:
        op_generator(op, g, d); pow_involutory(*d, g, p[0], m); return 0;
    case OP_SQRTX: case OP_SQRTY: case OP_SQRTW:
        op_generator(op, g, d); pow_involutory(*d, g, 0.5, m); return 0;
    case OP_FSIM: {
        double th = p[0], ph = p[1];
        mat_eye(4, m);
        m[5] = cos(th); m[6] = -I * sin(th);
        m[9] = -I * sin(th); m[10] = cos(th);
        m[15] = cexp(-I * ph);
        *d = 4; return 0; }
    case OP_MATRIX1: case OP_MATRIX2: {
        int dd = op == OP_MATRIX1 ? 2 : 4;
        for (int i = 0; i < dd * dd; i++) m[i] = explicit_m[2 * i] + I * explicit_m[2 * i + 1];
        *d = dd; return 0; }
    default:
        return 1;
    }
}

/* Derivative of the gate matrix with respect to its parameter `which`. */
static int gate_dmatrix(int op, const double *p, int which, cplx *dm, int *d)
{
    cplx g[16], m[16], t[16];
    switch (op) {
    case OP_RX: case OP_RY: case OP_RZ: case OP_RZZ:
        /* d/dtheta exp(-i theta G / 2) = (-i/2) G exp(-i theta G / 2) */
        op_generator(op, g, d); rot_involutory(*d, g, p[0], m);
        mat_mul(*d, g, m, t);
        for (int i = 0; i < *d * *d; i++) dm[i] = -0.5 * I * t[i];
        return 0;
    case OP_XPOW: case OP_YPOW: case OP_ZPOW: case OP_CZPOW: case OP_CNOTPOW:
    case OP_XXPOW: case OP_YYPOW: case OP_ZZPOW:
        /* G^t = exp(i pi t (I - G) / 2), so d/dt G^t = (i pi / 2)(I - G) G^t */
        op_generator(op, g, d); pow_involutory(*d, g, p[0], m);
        for (int i = 0; i < *d; i++)
            for (int j = 0; j < *d; j++) t[i * *d + j] = (i == j ? 1.0 : 0.0) - g[i * *d + j];
        mat_mul(*d, t, m, dm);
        for (int i = 0; i < *d * *d; i++) dm[i] *= 0.5 * M_PI * I;
        return 0;
    case OP_FSIM: {
        double th = p[0], ph = p[1];
        *d = 4;
        for (int i = 0; i < 16; i++) dm[i] = 0;
        if (which == 0) {
            dm[5] = -sin(th); dm[6] = -I * cos(th);
            dm[9] = -I * cos(th); dm[10] = -sin(th);
        } else {
            dm[15] = -I * cexp(-I * ph);
        }
        return 0; }
    default:
        return 1;
    }
}

/* ------------------------------------------------------------ containers */
typedef struct {
    int op, nq, np;
    int q[2];
    int sym[3];
    double scale[3], offset[3];
    int chan; /* OP_PCHAN: its ordinal among the circuit's channels */
    double mat[32];
    int *pq, *pp; /* OP_PAULIEXP: its nq qubits and their Paulis (1=X, 2=Y, 3=Z) */
} OGate;

typedef struct {
    int n, ngates;
    OGate *g;
} OCircuit;

typedef struct {
    int B, S, nmax;
    OCircuit *c;
} OProgram;

typedef struct {
    int nf;
    double coeff;
    int q[64];
    int pauli[64];
} OTerm;

typedef struct {
    int B, K;
    int *start; /* [B*K + 1] CSR offsets into terms */
    OTerm *t;
} OObs;

typedef struct {
    const uint8_t *p, *end;
    int bad;
} Rd;
static uint32_t rd_u32(Rd *r)
{
    uint32_t v = 0;
    if (r->end - r->p < 4) { r->bad = 1; return 0; }
    memcpy(&v, r->p, 4); r->p += 4; return v;
}
static uint16_t rd_u16(Rd *r)
{
    uint16_t v = 0;
    if (r->end - r->p < 2) { r->bad = 1; return 0; }
    memcpy(&v, r->p, 2); r->p += 2; return v;
}
static uint8_t rd_u8(Rd *r)
{
    if (r->end - r->p < 1) { r->bad = 1; return 0; }
    return *r->p++;
}
static double rd_f64(Rd *r)
{
    double v = 0;
    if (r->end - r->p < 8) { r->bad = 1; return 0; }
    memcpy(&v, r->p, 8); r->p += 8; return v;
}

void orc_program_free(void *h)
{
    OProgram *pr = (OProgram *)h;
    if (!pr) return;
    for (int b = 0; b < pr->B; b++) {
        for (int i = 0; i < pr->c[b].ngates; i++) {
            free(pr->c[b].g[i].pq);
            free(pr->c[b].g[i].pp);
        }
        free(pr->c[b].g);
    }
    free(pr->c);
    free(pr);
}

int orc_program_parse(const void *blob, size_t nbytes, void **out)
{
    Rd r = {(const uint8_t *)blob, (const uint8_t *)blob + nbytes, 0};
    if (nbytes < 16 || memcmp(blob, "TQP1", 4) != 0) return fail("bad program magic");
    r.p += 4;
    uint32_t ver = rd_u32(&r), B = rd_u32(&r), S = rd_u32(&r);
    if (ver != 1) return fail("bad program version");
    if (B > (1u << 24) || S > (1u << 24)) return fail("bad program header");
    OProgram *pr = calloc(1, sizeof *pr);
    pr->B = (int)B; pr->S = (int)S;
    pr->c = calloc(B ? B : 1, sizeof(OCircuit));
    for (uint32_t b = 0; b < B; b++) {
        uint32_t n = rd_u32(&r), ng = rd_u32(&r);
        if (r.bad || n > 34 || ng > (1u << 24)) { orc_program_free(pr); return fail("bad circuit header"); }
        OCircuit *c = &pr->c[b];
        int nchan = 0;
        c->n = (int)n; c->ngates = (int)ng;
        c->g = calloc(ng ? ng : 1, sizeof(OGate));
        if ((int)n > pr->nmax) pr->nmax = (int)n;
        for (uint32_t i = 0; i < ng; i++) {
            OGate *g = &c->g[i];
            g->op = rd_u16(&r); g->nq = rd_u8(&r); g->np = rd_u8(&r);
            if (!r.bad && g->op == OP_PAULIEXP) {
                /* w qubits (distinct), one parameter, then w Pauli codes */
                if (g->np != 1 || g->nq > (int)n) { orc_program_free(pr); return fail("bad Pauli exponential"); }
                g->pq = calloc(g->nq ? g->nq : 1, sizeof(int));
                g->pp = calloc(g->nq ? g->nq : 1, sizeof(int));
                for (int j = 0; j < g->nq; j++) {
                    uint32_t q = rd_u32(&r);
                    if (q >= n) { orc_program_free(pr); return fail("qubit out of range"); }
                    for (int k = 0; k < j; k++)
                        if (g->pq[k] == (int)q) { orc_program_free(pr); return fail("duplicate qubit"); }
                    g->pq[j] = (int)q;
                }
                int32_t s = (int32_t)rd_u32(&r);
                g->sym[0] = s; g->scale[0] = rd_f64(&r); g->offset[0] = rd_f64(&r);
                if (s < -1 || s >= (int32_t)S) { orc_program_free(pr); return fail("symbol out of range"); }
                for (int j = 0; j < g->nq; j++) {
                    g->pp[j] = rd_u8(&r);
                    if (g->pp[j] < 1 || g->pp[j] > 3) { orc_program_free(pr); return fail("bad Pauli code"); }
                }
                if (r.bad) { orc_program_free(pr); return fail("truncated program"); }
                continue;
            }
            int enq, enp;
            if (r.bad || op_arity(g->op, &enq, &enp) || enq != g->nq || enp != g->np) {
                orc_program_free(pr); return fail("bad gate opcode/arity");
            }
            for (int j = 0; j < g->nq; j++) {
                uint32_t q = rd_u32(&r);
                if (q >= n) { orc_program_free(pr); return fail("qubit out of range"); }
                g->q[j] = (int)q;
            }
            if (g->nq == 2 && g->q[0] == g->q[1]) { orc_program_free(pr); return fail("duplicate qubit"); }
            for (int j = 0; j < g->np; j++) {
                int32_t s = (int32_t)rd_u32(&r);
                g->sym[j] = s;
                g->scale[j] = rd_f64(&r);
                g->offset[j] = rd_f64(&r);
                if (s < -1 || s >= (int32_t)S) { orc_program_free(pr); return fail("symbol out of range"); }
            }
            if (g->op == OP_PCHAN) {
                double tot = 0;
                for (int j = 0; j < 3; j++) {
                    if (g->sym[j] != -1 || !(g->offset[j] >= 0.0)) {
                        orc_program_free(pr); return fail("channel probabilities must be constants >= 0");
                    }
                    tot += g->offset[j];
                }
                if (!(tot <= 1.0)) { orc_program_free(pr); return fail("channel probabilities sum above 1"); }
                g->chan = nchan++;
            }
            int nm = g->op == OP_MATRIX1 ? 8 : g->op == OP_MATRIX2 ? 32 : 0;
            for (int j = 0; j < nm; j++) g->mat[j] = rd_f64(&r);
            if (r.bad) { orc_program_free(pr); return fail("truncated program"); }
        }
    }
    if (r.p != r.end) { orc_program_free(pr); return fail("trailing bytes in program"); }
    *out = pr;
    return 0;
}

int orc_program_info(void *h, int *B, int *S, int *nmax, int *nq)
{
    OProgram *pr = (OProgram *)h;
    *B = pr->B; *S = pr->S; *nmax = pr->nmax;
    if (nq)
        for (int b = 0; b < pr->B; b++) nq[b] = pr->c[b].n;
    return 0;
}

void orc_obs_free(void *h)
{
    OObs *o = (OObs *)h;
    if (!o) return;
    free(o->start); free(o->t); free(o);
}

int orc_obs_parse(const void *blob, size_t nbytes, void **out)
{
    Rd r = {(const uint8_t *)blob, (const uint8_t *)blob + nbytes, 0};
    if (nbytes < 16 || memcmp(blob, "TQO1", 4) != 0) return fail("bad observable magic");
    r.p += 4;
    uint32_t ver = rd_u32(&r), B = rd_u32(&r), K = rd_u32(&r);
    if (ver != 1) return fail("bad observable version");
    if ((uint64_t)B * K > (1u << 26)) return fail("bad observable header");
    OObs *o = calloc(1, sizeof *o);
    o->B = (int)B; o->K = (int)K;
    o->start = calloc((size_t)B * K + 1, sizeof(int));
    size_t cap = 16, nt = 0;
    o->t = malloc(cap * sizeof(OTerm));
    for (size_t s = 0; s < (size_t)B * K; s++) {
        o->start[s] = (int)nt;
        uint32_t T = rd_u32(&r);
        if (r.bad || T > (1u << 24)) { orc_obs_free(o); return fail("bad term count"); }
        for (uint32_t t = 0; t < T; t++) {
            if (nt == cap) { cap *= 2; o->t = realloc(o->t, cap * sizeof(OTerm)); }
            OTerm *tm = &o->t[nt++];
            tm->coeff = rd_f64(&r);
            uint32_t nf = rd_u32(&r);
            if (r.bad || nf > 64) { orc_obs_free(o); return fail("bad factor count"); }
            tm->nf = (int)nf;
            for (uint32_t f = 0; f < nf; f++) {
                tm->q[f] = (int)rd_u32(&r);
                tm->pauli[f] = rd_u8(&r);
                if (tm->pauli[f] < 1 || tm->pauli[f] > 3) { orc_obs_free(o); return fail("bad pauli code"); }
                for (uint32_t e = 0; e < f; e++)
                    if (tm->q[e] == tm->q[f]) { orc_obs_free(o); return fail("duplicate qubit in term"); }
            }
            if (r.bad) { orc_obs_free(o); return fail("truncated observable"); }
        }
    }
    o->start[(size_t)B * K] = (int)nt;
    if (r.p != r.end) { orc_obs_free(o); return fail("trailing bytes in observable"); }
    *out = o;
    return 0;
}

/* -------------------------------------------------------- state kernels */
/* optional emulation of complex64 storage, for measuring the fp32 floor */
static int g_c64_storage = 0;
void orc_set_c64_storage(int on) { g_c64_storage = on; }

/* Apply a d x d matrix (d = 2^nq) to qubits qs of an n-qubit state: for every
 * index whose gate bits are all zero, gather the 2^nq amplitudes, multiply,
 * scatter back. */
static void apply_matrix(cplx *psi, int n, int nq, const int *qs, const cplx *m, int par)
{
    const int64_t N = (int64_t)1 << n;
    const int d = 1 << nq;
    int64_t bit[2] = {0, 0};
    for (int j = 0; j < nq; j++) bit[j] = (int64_t)1 << (n - 1 - qs[j]);
    int64_t gmask = bit[0] | bit[1];
#pragma omp parallel for if (par) schedule(static)
    for (int64_t i = 0; i < N; i++) {
        if (i & gmask) continue;
        int64_t idx[4];
        cplx v[4], w[4];
        for (int a = 0; a < d; a++) {
            int64_t k = i;
            for (int j = 0; j < nq; j++)
                if ((a >> (nq - 1 - j)) & 1) k |= bit[j];
            idx[a] = k;
            v[a] = psi[k];
        }
        for (int r = 0; r < d; r++) {
            cplx s = 0;
            for (int c = 0; c < d; c++) s += m[r * d + c] * v[c];
            w[r] = s;
        }
        for (int r = 0; r < d; r++) {
            if (g_c64_storage) w[r] = (float)creal(w[r]) + I * (float)cimag(w[r]);
            psi[idx[r]] = w[r];
        }
    }
}

/* psi <- a psi + b P psi for the Pauli string of an OP_PAULIEXP gate: with
 * (a, b) = (cos eta, -i sin eta) the gate exp(-i eta P) = cos(eta) I -
 * i sin(eta) P (Sec. "Quantum Neural Networks", eqs. Pauli_decomp and
 * cs_decomp), (cos eta, i sin eta) its inverse and (-sin eta, -i cos eta)
 * its derivative.  P psi: the string's 2x2 Paulis applied one by one. */
static void apply_pauli_exp(cplx *psi, int n, const OGate *g, cplx a, cplx b, int par)
{
    const int64_t N = (int64_t)1 << n;
    cplx *tmp = malloc(sizeof(cplx) * N);
    memcpy(tmp, psi, sizeof(cplx) * N);
    for (int f = 0; f < g->nq; f++) {
        cplx m[4];
        pauli2(g->pp[f], m);
        apply_matrix(tmp, n, 1, &g->pq[f], m, par);
    }
    for (int64_t i = 0; i < N; i++) {
        cplx w = a * psi[i] + b * tmp[i];
        if (g_c64_storage) w = (float)creal(w) + I * (float)cimag(w);
        psi[i] = w;
    }
    free(tmp);
}

static void dagger(int d, const cplx *m, cplx *out)
{
    for (int i = 0; i < d; i++)
        for (int j = 0; j < d; j++) out[j * d + i] = conj(m[i * d + j]);
}

/* eta = scale * theta[b, sym] + offset; constants (sym < 0) take the offset */
static void resolve(const OGate *g, const double *theta_row, double *eta)
{
    for (int j = 0; j < g->np; j++)
        eta[j] = g->sym[j] >= 0 ? g->scale[j] * theta_row[g->sym[j]] + g->offset[j] : g->offset[j];
}

/* ------------------------------------------------------------------ noise */
/* Trajectory simulation of noisy circuits (Sec. "Noise in qsim"): every row
 * is one trajectory; at each channel one Kraus operator is drawn and
 * applied.  For a Pauli channel (X, Y, Z with probabilities p_x, p_y, p_z,
 * else the identity) the draw of channel k of batch row b is
 * r = (u >> 11) 2^-53 with u = output number (b 2^32 + k) of SplitMix64 from
 * the noise seed: X if r < p_x, Y if r < p_x + p_y, Z if r < p_x + p_y + p_z
 * (sums in that order, in fp64), else I. */
static uint64_t g_noise_seed = 0;
void orc_set_noise_seed(uint64_t seed) { g_noise_seed = seed; }
/* added to a program row's index in the draws: rows of a larger batch
 * simulated one by one keep their own draws */
static int64_t g_row_offset = 0;
void orc_set_row_offset(int64_t off) { g_row_offset = off; }

uint64_t orc_splitmix64(uint64_t seed, uint64_t counter);

/* 0 = I, 1 = X, 2 = Y, 3 = Z */
int orc_channel_pick(uint64_t seed, int64_t row, int chan, double px, double py, double pz)
{
    const uint64_t u = orc_splitmix64(seed, ((uint64_t)row << 32) | (uint64_t)chan);
    const double r = (double)(u >> 11) * 0x1.0p-53;
    if (r < px) return 1;
    if (r < px + py) return 2;
    if (r < px + py + pz) return 3;
    return 0;
}

/* the Pauli a channel gate applies in row `row` (the identity as I) */
static void channel_matrix(const OGate *g, int64_t row, cplx *m)
{
    const int k = orc_channel_pick(g_noise_seed, row + g_row_offset, g->chan, g->offset[0], g->offset[1], g->offset[2]);
    if (k == 0) mat_eye(2, m);
    else pauli2(k, m);
}

/* psi = W_G ... W_1 |0..0> for one row; parameter `shift_param` of gate
 * `shift_gate` (none when negative) is taken at its resolved value plus
 * `delta` (the shifted circuits of the parameter-shift rule) */
static void simulate_row_shifted(const OCircuit *c, const double *theta_row, int64_t row, int shift_gate,
                                 int shift_param, double delta, cplx *psi, int par)
{
    const int64_t N = (int64_t)1 << c->n;
    for (int64_t i = 0; i < N; i++) psi[i] = 0;
    psi[0] = 1;
    for (int i = 0; i < c->ngates; i++) {
        const OGate *g = &c->g[i];
        double eta[3];
        cplx m[16];
        int d;
        resolve(g, theta_row, eta);
        if (i == shift_gate) eta[shift_param] += delta;
        if (g->op == OP_PAULIEXP) {
            apply_pauli_exp(psi, c->n, g, cos(eta[0]), -I * sin(eta[0]), par);
            continue;
        }
        if (g->op == OP_PCHAN) {
            channel_matrix(g, row, m);
            apply_matrix(psi, c->n, 1, g->q, m, par);
            continue;
        }
        gate_matrix(g->op, eta, g->mat, m, &d);
        apply_matrix(psi, c->n, g->nq, g->q, m, par);
    }
}

static void simulate_row(const OCircuit *c, const double *theta_row, int64_t row, cplx *psi, int par)
{
    simulate_row_shifted(c, theta_row, row, -1, 0, 0.0, psi, par);
}

/* out += coeff * P psi for one Pauli string term */
static void add_pauli_term(const OTerm *t, int n, const cplx *psi, cplx *tmp, cplx *out, cplx coeff, int par)
{
    const int64_t N = (int64_t)1 << n;
    memcpy(tmp, psi, sizeof(cplx) * N);
    for (int f = 0; f < t->nf; f++) {
        cplx m[4];
        pauli2(t->pauli[f], m);
        apply_matrix(tmp, n, 1, &t->q[f], m, par);
    }
    for (int64_t i = 0; i < N; i++) out[i] += coeff * tmp[i];
}

static cplx inner(const cplx *a, const cplx *b, int64_t N)
{
    cplx s = 0;
    for (int64_t i = 0; i < N; i++) s += conj(a[i]) * b[i];
    return s;
}

static int check_obs(const OProgram *pr, const OObs *o)
{
    if (o->B != pr->B) return fail("observable batch size differs from program");
    for (int b = 0; b < pr->B; b++)
        for (int k = 0; k < o->K; k++)
            for (int t = o->start[b * o->K + k]; t < o->start[b * o->K + k + 1]; t++)
                for (int f = 0; f < o->t[t].nf; f++)
                    if (o->t[t].q[f] >= pr->c[b].n) return fail("observable qubit out of range");
    return 0;
}

int orc_simulate_state(void *hp, const double *theta, double *out)
{
    OProgram *pr = (OProgram *)hp;
    const int64_t stride = (int64_t)1 << pr->nmax;
    int par = pr->B == 1;
#pragma omp parallel for if (!par) schedule(dynamic)
    for (int b = 0; b < pr->B; b++) {
        cplx *row = (cplx *)out + (int64_t)b * stride;
        for (int64_t i = 0; i < stride; i++) row[i] = 0;
        simulate_row(&pr->c[b], theta + (int64_t)b * pr->S, b, row, par);
    }
    return 0;
}

/* out[b,k] = Re <psi_b| h_{b,k} |psi_b>; imag (nullable) receives the
 * imaginary part, which is zero for Hermitian h up to rounding. */
int orc_expectation(void *hp, const double *theta, void *ho, double *out, double *imag)
{
    OProgram *pr = (OProgram *)hp;
    OObs *o = (OObs *)ho;
    if (check_obs(pr, o)) return 1;
    int par = pr->B == 1;
#pragma omp parallel for if (!par) schedule(dynamic)
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        const int64_t N = (int64_t)1 << c->n;
        cplx *psi = malloc(sizeof(cplx) * N), *tmp = malloc(sizeof(cplx) * N), *hp_ = malloc(sizeof(cplx) * N);
        simulate_row(c, theta + (int64_t)b * pr->S, b, psi, par);
        for (int k = 0; k < o->K; k++) {
            for (int64_t i = 0; i < N; i++) hp_[i] = 0;
            for (int t = o->start[b * o->K + k]; t < o->start[b * o->K + k + 1]; t++)
                add_pauli_term(&o->t[t], c->n, psi, tmp, hp_, o->t[t].coeff, par);
            cplx e = inner(psi, hp_, N);
            out[(int64_t)b * o->K + k] = creal(e);
            if (imag) imag[(int64_t)b * o->K + k] = cimag(e);
        }
        free(psi); free(tmp); free(hp_);
    }
    return 0;
}

/* ------------------------------------------------- sampled expectations */
/* Expectation estimated from samples (Sec. "Sampling and Expectation
 * Values": sample bitstrings in the measurement basis, apply the measurement
 * to each, average).  For h = sum_t c_t P_t each non-identity term is
 * measured `reps` times on its own: a shot of P_t yields +1 with probability
 * (1 + <P_t>)/2, else -1 (the parity of the term's qubits after rotating them
 * to the Z basis), and the estimate is sum_t c_t (2 n_t / reps - 1) plus the
 * identity terms' coefficients, n_t the number of +1 shots.  Shot s of term
 * t of observable k in batch row b is +1 when (u >> 11) 2^-53 < q with
 * q = (1 + e_t)/2 in fp64 (e_t clamped to [-1, 1]) and u the output number
 * ((b K + k) 2^40 + t 2^24 + s) of SplitMix64 started at `seed`. */
static uint64_t sampled_count(uint64_t seed, int64_t bk, int t, int reps, double e)
{
    if (e > 1.0) e = 1.0;
    if (e < -1.0) e = -1.0;
    const double q = 0.5 * (1.0 + e);
    uint64_t n = 0;
    for (int s = 0; s < reps; s++) {
        const uint64_t u = orc_splitmix64(seed, ((uint64_t)bk << 40) | ((uint64_t)t << 24) | (uint64_t)s);
        n += ((double)(u >> 11) * 0x1.0p-53 < q);
    }
    return n;
}

static int check_sampled(const OObs *o, int reps)
{
    if (reps < 1 || reps >= (1 << 24)) return fail("repetitions must be in [1, 2^24)");
    if ((int64_t)o->B * o->K >= ((int64_t)1 << 24)) return fail("too many (row, observable) pairs for the shot counter");
    for (int i = 0; i < o->B * o->K; i++)
        if (o->start[i + 1] - o->start[i] >= (1 << 16)) return fail("too many terms in one observable");
    return 0;
}

/* full pipeline: exact term expectations from the complex128 state */
int orc_sampled_expectation(void *hp, const double *theta, void *ho, int reps, uint64_t seed, double *out)
{
    OProgram *pr = (OProgram *)hp;
    OObs *o = (OObs *)ho;
    if (check_obs(pr, o) || check_sampled(o, reps)) return 1;
    int par = pr->B == 1;
#pragma omp parallel for if (!par) schedule(dynamic)
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        const int64_t N = (int64_t)1 << c->n;
        cplx *psi = malloc(sizeof(cplx) * N), *tmp = malloc(sizeof(cplx) * N), *hp_ = malloc(sizeof(cplx) * N);
        simulate_row(c, theta + (int64_t)b * pr->S, b, psi, par);
        for (int k = 0; k < o->K; k++) {
            double est = 0.0;
            const int t0 = o->start[b * o->K + k], t1 = o->start[b * o->K + k + 1];
            for (int t = t0; t < t1; t++) {
                const OTerm *tm = &o->t[t];
                if (tm->nf == 0) { est += tm->coeff; continue; }
                for (int64_t i = 0; i < N; i++) hp_[i] = 0;
                add_pauli_term(tm, c->n, psi, tmp, hp_, 1.0, par);
                const double e = creal(inner(psi, hp_, N));
                const uint64_t n = sampled_count(seed, (int64_t)b * o->K + k, t - t0, reps, e);
                est += tm->coeff * (2.0 * (double)n / reps - 1.0);
            }
            out[(int64_t)b * o->K + k] = est;
        }
        free(psi); free(tmp); free(hp_);
    }
    return 0;
}

/* the same estimate from given term expectations: term_exp[b, j] for the
 * j-th non-identity term of row b over (k, t) in order, Kt per row */
int orc_sampled_from_terms(void *ho, const float *term_exp, int Kt, int reps, uint64_t seed, double *out)
{
    OObs *o = (OObs *)ho;
    if (check_sampled(o, reps)) return 1;
    for (int b = 0; b < o->B; b++) {
        int j = 0;
        for (int k = 0; k < o->K; k++) {
            double est = 0.0;
            const int t0 = o->start[b * o->K + k], t1 = o->start[b * o->K + k + 1];
            for (int t = t0; t < t1; t++) {
                const OTerm *tm = &o->t[t];
                if (tm->nf == 0) { est += tm->coeff; continue; }
                if (j >= Kt) return fail("term_exp has fewer terms than the observables");
                const uint64_t n = sampled_count(seed, (int64_t)b * o->K + k, t - t0, reps,
                                                 (double)term_exp[(int64_t)b * Kt + j++]);
                est += tm->coeff * (2.0 * (double)n / reps - 1.0);
            }
            out[(int64_t)b * o->K + k] = est;
        }
    }
    return 0;
}

/* ------------------------------------------ shift and difference rules */
/* The two-term parameter-shift rule of parameter j of a gate (Sec.
 * "Parameter shift methods", eq. parshift_grad): when the parameter enters
 * as exp(-i eta G) with G of two distinct eigenvalues e0 < e1, every
 * expectation is a + b cos(r eta) + c sin(r eta) with r = e1 - e0, so
 * f'(eta) = (r / 2) (f(eta + pi / (2 r)) - f(eta - pi / (2 r))).
 *   RX, RY, RZ, RZZ = exp(-i eta G / 2), G involutory: r = 1.
 *   pow gates G^t = e^{i pi t / 2} exp(-i (pi t / 2) G): r = pi (in t).
 *   exp(-i eta P) of a Pauli string: r = 2, the printed rule with pi / 4.
 *   fSim's phi, exp(-i phi |11><11|): r = 1.
 * fSim's theta, exp(-i theta (XX + YY) / 2), has three eigenvalues and no
 * two-term rule; it returns 1. */
static int shift_rule(int op, int j, double *delta, double *factor)
{
    switch (op) {
    case OP_RX: case OP_RY: case OP_RZ: case OP_RZZ:
        *delta = M_PI / 2.0; *factor = 0.5; return 0;
    case OP_XPOW: case OP_YPOW: case OP_ZPOW: case OP_CZPOW: case OP_CNOTPOW:
    case OP_XXPOW: case OP_YYPOW: case OP_ZZPOW:
        *delta = 0.5; *factor = M_PI / 2.0; return 0;
    case OP_PAULIEXP:
        *delta = M_PI / 4.0; *factor = 1.0; return 0;
    case OP_FSIM:
        if (j == 1) { *delta = M_PI / 2.0; *factor = 0.5; return 0; }
        return 1;
    default:
        return 1;
    }
}

/* number of symbolic parameters (shift-rule occurrences) of a circuit */
static int count_occurrences(const OCircuit *c)
{
    int n = 0;
    for (int i = 0; i < c->ngates; i++)
        for (int j = 0; j < c->g[i].np; j++) n += c->g[i].sym[j] >= 0;
    return n;
}

/* The K values of row b's observables on state psi: exact (reps = 0), or
 * estimated from reps shots per non-identity term with the shot counter of
 * (row e, observable k) as in the sampled expectation above. */
static void observable_values(const OObs *o, int b, int n, const cplx *psi, cplx *tmp, cplx *hp_, int reps,
                              uint64_t seed, int64_t e, double *out, int par)
{
    const int64_t N = (int64_t)1 << n;
    for (int k = 0; k < o->K; k++) {
        double v = 0.0;
        const int t0 = o->start[b * o->K + k], t1 = o->start[b * o->K + k + 1];
        for (int t = t0; t < t1; t++) {
            const OTerm *tm = &o->t[t];
            if (tm->nf == 0) { v += tm->coeff; continue; }
            for (int64_t i = 0; i < N; i++) hp_[i] = 0;
            add_pauli_term(tm, n, psi, tmp, hp_, 1.0, par);
            const double pe = creal(inner(psi, hp_, N));
            if (reps == 0) v += tm->coeff * pe;
            else v += tm->coeff * (2.0 * (double)sampled_count(seed, e * o->K + k, t - t0, reps, pe) / reps - 1.0);
        }
        out[k] = v;
    }
}

/* Gradients of sum_k g_{b,k} <h_{b,k}> by the parameter-shift rule: every
 * symbolic parameter (occurrence) of a circuit is shifted by +-delta alone,
 * the circuit re-simulated, and grad[b, sym] += scale * factor *
 * sum_k g_k (f_k(+) - f_k(-)) (shared symbols add over their occurrences,
 * eq. chain_rule).  With reps > 0 each shifted circuit's expectations are
 * sampled estimates: the shifted circuits form a batch of sum_b 2 O_b rows
 * (O_b the occurrences of row b) in the order (row, occurrence in gate and
 * parameter order, + before -), and shifted circuit e draws its shots with
 * the counter of row e. */
int orc_param_shift_grad(void *hp, const double *theta, void *ho, const double *upstream, int reps, uint64_t seed,
                         double *grad)
{
    OProgram *pr = (OProgram *)hp;
    OObs *o = (OObs *)ho;
    if (check_obs(pr, o)) return 1;
    if (reps < 0) return fail("repetitions must be >= 0");
    int64_t *ebase = malloc(sizeof(int64_t) * (pr->B + 1));
    ebase[0] = 0;
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        for (int i = 0; i < c->ngates; i++)
            for (int j = 0; j < c->g[i].np; j++) {
                double dl, fc;
                if (c->g[i].sym[j] >= 0 && shift_rule(c->g[i].op, j, &dl, &fc)) {
                    free(ebase);
                    return fail("a symbolic parameter has no two-term shift rule (fSim theta)");
                }
            }
        ebase[b + 1] = ebase[b] + 2 * (int64_t)count_occurrences(c);
    }
    if (reps > 0) {
        if (reps >= (1 << 24)) { free(ebase); return fail("repetitions must be in [1, 2^24)"); }
        if (ebase[pr->B] * o->K >= ((int64_t)1 << 24)) {
            free(ebase);
            return fail("too many (shifted circuit, observable) pairs for the shot counter");
        }
        if (check_sampled(o, reps)) { free(ebase); return 1; }
    }
    int par = pr->B == 1;
#pragma omp parallel for if (!par) schedule(dynamic)
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        const double *th = theta + (int64_t)b * pr->S;
        double *gr = grad + (int64_t)b * pr->S;
        const int64_t N = (int64_t)1 << c->n;
        cplx *psi = malloc(sizeof(cplx) * N), *tmp = malloc(sizeof(cplx) * N), *hp_ = malloc(sizeof(cplx) * N);
        double *fp = malloc(sizeof(double) * (o->K + 1)), *fm = malloc(sizeof(double) * (o->K + 1));
        for (int s = 0; s < pr->S; s++) gr[s] = 0;
        int64_t occ = 0;
        for (int i = 0; i < c->ngates; i++) {
            const OGate *g = &c->g[i];
            for (int j = 0; j < g->np; j++) {
                if (g->sym[j] < 0) continue;
                double dl, fc;
                shift_rule(g->op, j, &dl, &fc);
                const int64_t e = ebase[b] + 2 * occ++;
                simulate_row_shifted(c, th, b, i, j, dl, psi, par);
                observable_values(o, b, c->n, psi, tmp, hp_, reps, seed, e, fp, par);
                simulate_row_shifted(c, th, b, i, j, -dl, psi, par);
                observable_values(o, b, c->n, psi, tmp, hp_, reps, seed, e + 1, fm, par);
                double d = 0.0;
                for (int k = 0; k < o->K; k++) d += upstream[(int64_t)b * o->K + k] * (fp[k] - fm[k]);
                gr[g->sym[j]] += g->scale[j] * fc * d;
            }
        }
        free(psi); free(tmp); free(hp_); free(fp); free(fm);
    }
    free(ebase);
    return 0;
}

/* Gradients by central finite differences in the symbol values (Sec.
 * "Finite difference methods", eq. central_diff):
 * grad[b, s] = sum_k g_{b,k} (f_k(theta + eps e_s) - f_k(theta - eps e_s)) / (2 eps),
 * the shifted symbol value formed in fp64.  Every symbol is shifted; one no
 * gate of the row uses gets exactly 0. */
int orc_finite_diff_grad(void *hp, const double *theta, void *ho, const double *upstream, double eps, double *grad)
{
    OProgram *pr = (OProgram *)hp;
    OObs *o = (OObs *)ho;
    if (check_obs(pr, o)) return 1;
    if (!(eps > 0.0)) return fail("eps must be > 0");
    int par = pr->B == 1;
#pragma omp parallel for if (!par) schedule(dynamic)
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        const int64_t N = (int64_t)1 << c->n;
        cplx *psi = malloc(sizeof(cplx) * N), *tmp = malloc(sizeof(cplx) * N), *hp_ = malloc(sizeof(cplx) * N);
        double *fp = malloc(sizeof(double) * (o->K + 1)), *fm = malloc(sizeof(double) * (o->K + 1));
        double *th = malloc(sizeof(double) * (pr->S + 1));
        for (int s = 0; s < pr->S; s++) th[s] = theta[(int64_t)b * pr->S + s];
        for (int s = 0; s < pr->S; s++) {
            const double t0 = th[s];
            th[s] = t0 + eps;
            simulate_row(c, th, b, psi, par);
            observable_values(o, b, c->n, psi, tmp, hp_, 0, 0, 0, fp, par);
            th[s] = t0 - eps;
            simulate_row(c, th, b, psi, par);
            observable_values(o, b, c->n, psi, tmp, hp_, 0, 0, 0, fm, par);
            th[s] = t0;
            double d = 0.0;
            for (int k = 0; k < o->K; k++) d += upstream[(int64_t)b * o->K + k] * (fp[k] - fm[k]);
            grad[(int64_t)b * pr->S + s] = d / (2.0 * eps);
        }
        free(psi); free(tmp); free(hp_); free(fp); free(fm); free(th);
    }
    return 0;
}

/* Adjoint method: phi = H_g psi with H_g = sum_k g_k h_k; then for the gates
 * in reverse order: psi <- W^dagger psi; for every symbolic parameter,
 * grad[sym] += scale * 2 Re <phi| dW/deta |psi>; phi <- W^dagger phi. */
int orc_adjoint_grad(void *hp, const double *theta, void *ho, const double *upstream, double *grad)
{
    OProgram *pr = (OProgram *)hp;
    OObs *o = (OObs *)ho;
    if (check_obs(pr, o)) return 1;
    int par = pr->B == 1;
#pragma omp parallel for if (!par) schedule(dynamic)
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        const double *th = theta + (int64_t)b * pr->S;
        double *gr = grad + (int64_t)b * pr->S;
        const int64_t N = (int64_t)1 << c->n;
        cplx *psi = malloc(sizeof(cplx) * N), *phi = malloc(sizeof(cplx) * N);
        cplx *tmp = malloc(sizeof(cplx) * N), *dpsi = malloc(sizeof(cplx) * N);
        for (int s = 0; s < pr->S; s++) gr[s] = 0;
        simulate_row(c, th, b, psi, par);
        for (int64_t i = 0; i < N; i++) phi[i] = 0;
        for (int k = 0; k < o->K; k++) {
            double gk = upstream[(int64_t)b * o->K + k];
            for (int t = o->start[b * o->K + k]; t < o->start[b * o->K + k + 1]; t++)
                add_pauli_term(&o->t[t], c->n, psi, tmp, phi, gk * o->t[t].coeff, par);
        }
        for (int i = c->ngates - 1; i >= 0; i--) {
            const OGate *g = &c->g[i];
            double eta[3];
            cplx m[16], md[16];
            int d;
            resolve(g, th, eta);
            if (g->op == OP_PCHAN) { /* the trajectory's Pauli: its own inverse, no parameter */
                channel_matrix(g, b, m);
                apply_matrix(psi, c->n, 1, g->q, m, par);
                apply_matrix(phi, c->n, 1, g->q, m, par);
                continue;
            }
            if (g->op == OP_PAULIEXP) {
                const double cs = cos(eta[0]), sn = sin(eta[0]);
                apply_pauli_exp(psi, c->n, g, cs, I * sn, par);
                if (g->sym[0] >= 0) {
                    memcpy(dpsi, psi, sizeof(cplx) * N);
                    apply_pauli_exp(dpsi, c->n, g, -sn, -I * cs, par);
                    gr[g->sym[0]] += g->scale[0] * 2.0 * creal(inner(phi, dpsi, N));
                }
                apply_pauli_exp(phi, c->n, g, cs, I * sn, par);
                continue;
            }
            gate_matrix(g->op, eta, g->mat, m, &d);
            dagger(d, m, md);
            apply_matrix(psi, c->n, g->nq, g->q, md, par);
            for (int j = 0; j < g->np; j++) {
                if (g->sym[j] < 0) continue;
                cplx dm[16];
                gate_dmatrix(g->op, eta, j, dm, &d);
                memcpy(dpsi, psi, sizeof(cplx) * N);
                apply_matrix(dpsi, c->n, g->nq, g->q, dm, par);
                gr[g->sym[j]] += g->scale[j] * 2.0 * creal(inner(phi, dpsi, N));
            }
            apply_matrix(phi, c->n, g->nq, g->q, md, par);
        }
        free(psi); free(phi); free(tmp); free(dpsi);
    }
    return 0;
}

/* amplitudes <x_{b,m}| psi_b> at the given bitstrings (external convention) */
int orc_amplitudes(void *hp, const double *theta, const uint64_t *bits, int64_t M, double *out)
{
    OProgram *pr = (OProgram *)hp;
    for (int b = 0; b < pr->B; b++)
        for (int64_t m = 0; m < M; m++)
            if (bits[b * M + m] >> pr->c[b].n) return fail("bitstring out of range");
    int par = pr->B == 1;
#pragma omp parallel for if (!par) schedule(dynamic)
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        cplx *psi = malloc(sizeof(cplx) * ((int64_t)1 << c->n));
        simulate_row(c, theta + (int64_t)b * pr->S, b, psi, par);
        for (int64_t m = 0; m < M; m++) {
            cplx a = psi[bits[b * M + m]];
            out[2 * (b * M + m)] = creal(a);
            out[2 * (b * M + m) + 1] = cimag(a);
        }
        free(psi);
    }
    return 0;
}

/* ---------------------------------------------------------------- sampling */
/* SplitMix64 (Steele, Lea, Flood 2014): the output number `counter` of the
 * sequence whose state starts at `seed`; the state advances by the golden
 * gamma before every output. */
uint64_t orc_splitmix64(uint64_t seed, uint64_t counter)
{
    uint64_t z = seed + (counter + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Integer fixed-point inverse-CDF sampling of one row from its probabilities:
 * w_i = floor(p_i * 2^62), W = sum w_i, r_k = floor(u_k * W / 2^64), and shot k
 * is the unique i with C_i <= r_k < C_i + w_i (C = exclusive prefix of w).
 * A row with W = 0 has no distribution to draw from; every shot of it is the
 * marker 2^64 - 1 (no bitstring of at most 34 qubits takes that value). */
static int sample_row_from_p(const double *p, int64_t N, int64_t row, int64_t n_shots, uint64_t seed,
                             uint64_t *out)
{
    uint64_t *C = malloc(sizeof(uint64_t) * (N + 1));
    C[0] = 0;
    for (int64_t i = 0; i < N; i++) C[i + 1] = C[i] + (uint64_t)(p[i] * 0x1p62);
    uint64_t W = C[N];
    if (W == 0) {
        for (int64_t k = 0; k < n_shots; k++) out[k] = ~(uint64_t)0;
        free(C);
        return 0;
    }
    for (int64_t k = 0; k < n_shots; k++) {
        uint64_t u = orc_splitmix64(seed, (uint64_t)(row * n_shots + k));
        uint64_t r = (uint64_t)(((unsigned __int128)u * W) >> 64);
        /* largest i with C[i] <= r; since r < W, w_i > 0 at that i */
        int64_t lo = 0, hi = N; /* invariant: C[lo] <= r < C[hi] */
        while (hi - lo > 1) {
            int64_t mid = lo + (hi - lo) / 2;
            if (C[mid] <= r) lo = mid; else hi = mid;
        }
        out[k] = (uint64_t)lo;
    }
    free(C);
    return 0;
}

/* sample from given complex64 states [B, 2^n] (interleaved float re, im) */
int orc_sample_from_state(const float *state, int B, int n, int64_t n_shots, uint64_t seed, uint64_t *out)
{
    const int64_t N = (int64_t)1 << n;
    int bad = 0;
    for (int b = 0; b < B; b++) {
        double *p = malloc(sizeof(double) * N);
        const float *row = state + 2 * (int64_t)b * N;
#pragma omp parallel for if (B == 1) schedule(static)
        for (int64_t i = 0; i < N; i++) {
            double re = row[2 * i], im = row[2 * i + 1];
            p[i] = re * re + im * im;
        }
        bad |= sample_row_from_p(p, N, b, n_shots, seed, out + (int64_t)b * n_shots);
        free(p);
    }
    return bad ? fail("sampling failed") : 0;
}

/* full pipeline: simulate in complex128, then sample each row from its p */
int orc_sample(void *hp, const double *theta, int64_t n_shots, uint64_t seed, uint64_t *out)
{
    OProgram *pr = (OProgram *)hp;
    int par = pr->B == 1, bad = 0;
    for (int b = 0; b < pr->B; b++) {
        const OCircuit *c = &pr->c[b];
        const int64_t N = (int64_t)1 << c->n;
        cplx *psi = malloc(sizeof(cplx) * N);
        double *p = malloc(sizeof(double) * N);
        simulate_row(c, theta + (int64_t)b * pr->S, b, psi, par);
        for (int64_t i = 0; i < N; i++) p[i] = creal(psi[i]) * creal(psi[i]) + cimag(psi[i]) * cimag(psi[i]);
        bad |= sample_row_from_p(p, N, b, n_shots, seed, out + (int64_t)b * n_shots);
        free(psi); free(p);
    }
    return bad ? fail("sampling failed") : 0;
}

/* -------------------------------------------------- gate table accessors */
int orc_gate_matrix(int op, const double *params, const double *explicit_m, double *out, int *d)
{
    cplx m[16];
    if (op < 1 || op > OP_LAST || gate_matrix(op, params, explicit_m, m, d)) return fail("bad opcode");
    for (int i = 0; i < *d * *d; i++) { out[2 * i] = creal(m[i]); out[2 * i + 1] = cimag(m[i]); }
    return 0;
}

int orc_gate_dmatrix(int op, const double *params, int which, double *out, int *d)
{
    cplx m[16];
    if (op < 1 || op > OP_LAST || gate_dmatrix(op, params, which, m, d)) return fail("no derivative for opcode");
    for (int i = 0; i < *d * *d; i++) { out[2 * i] = creal(m[i]); out[2 * i + 1] = cimag(m[i]); }
    return 0;
}

int orc_op_arity(int op, int *nq, int *np) { return op_arity(op, nq, np); }
