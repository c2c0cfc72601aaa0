/*
 * tq.h -- C ABI of the batched state-vector simulation library for MI355X.
 *
 * The library runs the circuit-execution hot path of TensorFlow Quantum
 * (arXiv:2003.02989) on one AMD Instinct MI355X: batched state-vector
 * simulation of parameterized circuits in complex64, Pauli-sum expectation
 * values, bitstring sampling and adjoint-method gradients; noisy circuits as
 * trajectories (Pauli channels), expectations estimated from measurement
 * shots, and parameter-shift and finite-difference gradients as batched
 * launches.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Circuits and Pauli sums arrive as flat little-endian blobs (format in
 *    the description of tq_program_create / tq_observables_create).  A batch
 *    may mix circuits of different structure and qubit count (the paper's
 *    ops accept any batch of circuits, Sec. "Sampling and Expectation
 *    Values").
 *  - Qubit q of an n-qubit circuit is bit (n-1-q) of an amplitude index and
 *    of a sampled bitstring: qubit 0 is the most significant bit.
 *  - Every array argument of the compute calls is a DEVICE pointer owned by
 *    the caller, and `stream` is a hipStream_t (NULL = the null stream).
 *    Compute calls only enqueue work on `stream` and return without a host
 *    synchronisation; inputs and outputs must stay alive until the caller
 *    synchronises the stream.  Faults of enqueued kernels surface at that
 *    synchronisation.
 *  - All validation happens on the host, before anything is enqueued.  On an
 *    error the outputs are untouched, the call returns a non-zero tq_status
 *    and tq_last_error() returns a message (thread local).
 *  - The library owns only its internal workspaces (intermediate states,
 *    partial sums, fused gate matrices, sampler levels).  They are allocated
 *    on the device that is current at the first compute call, cached in the
 *    program handle and freed by tq_program_destroy.
 *  - Calls on distinct program handles may run from different threads; one
 *    handle must be used by one thread at a time, and concurrent calls on the
 *    same handle on different streams race on its workspaces.
 *  - No C++ exception crosses this boundary.
 */
#ifndef TQ_H
#define TQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tq_program_s *tq_program;
typedef struct tq_observables_s *tq_observables;

typedef enum {
    TQ_OK = 0,
    TQ_E_INVALID = 1,     /* malformed blob or argument: bad magic/version, qubit out of range or repeated,
                             symbol column >= S, observable qubit >= n_b, null pointer, negative size */
    TQ_E_UNSUPPORTED = 2, /* unknown opcode, or a problem outside the library's limits (n > 32) */
    TQ_E_NOMEM = 3,       /* a device workspace could not be allocated */
    TQ_E_DEVICE = 4       /* a HIP runtime error; its text is in tq_last_error() */
} tq_status;

/* Planner options; a zero field selects the default.
 *   max_tile_qubits: log2 of the amplitudes one workgroup stages in LDS per
 *                    forward pass (default 12, or 13 with specialize = 1;
 *                    allowed 8..13);
 *   low_qubits:      contiguous low index bits every tile keeps, so that each
 *                    wavefront reads runs of 2^low_qubits amplitudes
 *                    (default 6, allowed 3..8);
 *   fuse:            1 = fuse neighbouring gates into one matrix (default),
 *                    -1 = apply every gate on its own;
 *   max_pass_gates:  at most this many gates per sweep over the state
 *                    (default 0 = no limit; 1 makes every gate its own pass,
 *                    which measures the bandwidth of single-gate passes);
 *   specialize:      1 = every circuit structure runs kernels generated
 *                    for it (the resident kernel, or its forward and reverse
 *                    tile passes) and compiled with hipRTC on first use (or
 *                    by tq_program_specialize), with every stage and op
 *                    written in as constants; likewise an observable set that
 *                    is the same on every row (at most 16 observables and 64
 *                    terms, some with X or Y factors) gets expectation passes
 *                    generated for its terms, and a single observable that is
 *                    the same on every row (at most 1024 terms, states of more
 *                    than 12 qubits) gets passes generated for the adjoint's
 *                    phi = g H psi and its expectation.  Structures without
 *                    symbolic parameters get no generated reverse passes.
 *                    0 = the precompiled kernels that read the plan from
 *                    tables (default). */
typedef struct {
    int32_t max_tile_qubits;
    int32_t low_qubits;
    int32_t fuse;
    int32_t max_pass_gates;
    int32_t specialize;
} tq_options;

/* Parse, validate and plan a batch of B parameterized circuits over S symbols
 * (host only; no device call).  Blob:
 *     "TQP1" u32 version(=1) u32 B u32 S
 *     per circuit: u32 n_qubits u32 n_gates
 *       per gate:  u16 opcode u8 nq u8 np u32 qubit[nq]
 *                  np x { i32 symbol (-1 = constant) f64 scale f64 offset }
 *                  then 8 f64 for MATRIX1, 32 f64 for MATRIX2 (re, im, row major),
 *                  nq u8 Pauli codes (1 X, 2 Y, 3 Z) for PAULIEXP
 * A parameter resolves to eta = scale * symbol_values[b, symbol] + offset, the
 * affine symbol maps of the paper's chain rule (Sec. "Parameter shift
 * methods", eq. chain_rule); constants take eta = offset.
 * Opcodes (Cirq's gate set as the paper uses it; pow gates G^t follow the
 * phase convention G^t = e^{i pi t/2} (cos(pi t/2) I - i sin(pi t/2) G)):
 *     1 H  2 X  3 Y  4 Z  5 RX(theta)  6 RY  7 RZ  8 XPOW(t)  9 YPOW  10 ZPOW
 *     11 CZ  12 CNOT(control, target)  13 CZPOW(t)  14 CNOTPOW(t)  15 XXPOW(t)
 *     16 YYPOW(t)  17 ZZPOW(t)  18 RZZ(gamma) = exp(-i gamma Z Z / 2)
 *     19 SQRTX  20 SQRTY  21 SQRTW  22 FSIM(theta, phi)  23 MATRIX1
 *     24 MATRIX2  25 SWAP
 *     26 PAULIEXP(eta) = exp(-i eta P) = cos(eta) I - i sin(eta) P for the
 *        Pauli string P over its nq distinct qubits, any weight (nq = 0: the
 *        global phase exp(-i eta)); the exponentials of a generator's Pauli
 *        decomposition (Sec. "Quantum Neural Networks", eqs. Pauli_decomp and
 *        cs_decomp).  It is lowered to the gates above when the program is
 *        parsed (basis changes, a CNOT ladder around RZ / RZZ(2 eta)), so
 *        tq_program_describe counts the lowered gates.
 *     27 PCHAN(p_x, p_y, p_z), one qubit: a Pauli channel, X, Y or Z with these
 *        probabilities (constant parameters, each >= 0, sum <= 1), else the
 *        identity.  Noisy circuits run as trajectories (Sec. "Noise in
 *        qsim"): in every call each batch row draws one Pauli per channel and
 *        is then a pure circuit, so R rows holding the same circuit are R
 *        trajectories of it; tq_row_mean averages their outputs.  The draw of
 *        channel k (its ordinal among the circuit's channels) in batch row b:
 *        r = (u >> 11) 2^-53 with u the output number (b 2^32 + k) of
 *        SplitMix64 started at the program's noise seed
 *        (tq_program_set_noise_seed, default 0); X if r < p_x, Y if
 *        r < p_x + p_y, Z if r < p_x + p_y + p_z (fp64, in that order).
 * A two-qubit gate on (a, b) uses the local index 2*bit(a) + bit(b).
 * Circuits may have 0..32 qubits and any number of gates.  `opt` may be NULL.
 * On success *out owns the parsed program; release it with
 * tq_program_destroy. */
tq_status tq_program_create(const void *blob, size_t nbytes, const tq_options *opt, tq_program *out);
void tq_program_destroy(tq_program prog);

/* Seed of the channels' Kraus draws (opcode 27) in the program's later calls;
 * a new seed per call gives new trajectories.  Host only. */
tq_status tq_program_set_noise_seed(tq_program prog, uint64_t seed);

/* out[g, k] = (1/R) sum_{r < R} in[g R + r, k] for g < groups, k < K: the
 * average over R consecutive rows (the trajectories of one noisy circuit),
 * summed in fp64 in row order.  in: device float[groups R, K]; out: device
 * float[groups, K]; both caller-owned; enqueued on `stream`.  TQ_E_INVALID
 * for R < 1, negative sizes or NULL pointers with work to do. */
tq_status tq_row_mean(const float *in, int64_t groups, int32_t R, int32_t K, float *out, void *stream);

/* Compile the kernels a program created with specialize = 1 generates for
 * its circuit structures (per structure: the resident kernel when its
 * circuits run resident, else its forward and reverse tile passes), ahead of
 * their first launch.
 * target NULL: for the current device (the kernels are cached until the
 * process ends); otherwise an offload target such as "gfx950", for which the
 * code is only compiled and checked (no device is needed).  A compiler
 * failure returns TQ_E_DEVICE with the compiler's log in tq_last_error(); a
 * program without specialize = 1 returns TQ_OK at once. */
tq_status tq_program_specialize(tq_program prog, const char *target);

/* Batch size, symbol count, largest qubit count, and (when not NULL) the
 * qubit count of every circuit into qubits_per_circuit[B] (host memory). */
tq_status tq_program_info(tq_program prog, int32_t *B, int32_t *S, int32_t *max_qubits,
                          int32_t *qubits_per_circuit);

/* Parse B x K Pauli sums h_{b,k} = sum_t c_t P_t (Sec. "Sampling and
 * Expectations", eq. cost_lincomb).  Blob:
 *     "TQO1" u32 version(=1) u32 B u32 K
 *     per (b, k), row major: u32 T
 *       per term: f64 coeff u32 n_factors n_factors x { u32 qubit u8 pauli (1=X 2=Y 3=Z) }
 * An empty factor list is the identity term.  A qubit may appear once per
 * term; qubit ranges are checked against a program when both are used. */
tq_status tq_observables_create(const void *blob, size_t nbytes, tq_observables *out);
void tq_observables_destroy(tq_observables obs);
tq_status tq_observables_info(tq_observables obs, int32_t *B, int32_t *K);

/* Final state of every circuit (the paper's state op, Sec. "TFQ
 * architecture"): psi_b = W_G(eta_G) ... W_1(eta_1) |0...0>.
 * symbol_values: float32 [B, S] row major (may be NULL when S = 0).
 * states: complex64 [B, 2^max_qubits] (interleaved re, im); row b holds
 * 2^{n_b} amplitudes followed by zeros. */
tq_status tq_simulate_state(tq_program prog, const float *symbol_values, void *states, void *stream);

/* Expectation values out[b, k] = <psi_b| h_{b,k} |psi_b> (Sec. "Sampling and
 * Expectations", eq. qee_lincomb), float32 [B, K].  The imaginary part, zero
 * for Hermitian h, is dropped. */
tq_status tq_expectation(tq_program prog, const float *symbol_values, tq_observables obs, float *out,
                         void *stream);

/* n_shots bitstrings per circuit drawn from |psi_b,i|^2 (Sec. "Sampling and
 * Expectation Values"), uint64 [B, n_shots], bitstring i packed with qubit q at
 * bit n_b-1-q.  Rule (integer, order independent): p_i = re^2 + im^2 of the
 * complex64 amplitude in float64, w_i = floor(p_i 2^62), W = sum_i w_i,
 * u_k = SplitMix64 output number (b * n_shots + k) of the stream started at
 * `seed`, r_k = floor(u_k W / 2^64), and shot k is the unique i with
 * C_i <= r_k < C_i + w_i where C is the exclusive prefix sum of w.
 * n_shots >= 0.  A row with W = 0 (no distribution: an all-zero state)
 * yields 2^64 - 1 for every shot, a value no bitstring of at most 32 qubits
 * takes. */
tq_status tq_sample(tq_program prog, const float *symbol_values, int64_t n_shots, uint64_t seed,
                    uint64_t *out, void *stream);

/* One simulation serving both outputs of a random-circuit benchmark: the
 * samples of tq_sample (out, uint64 [B, n_shots], when n_shots > 0) and the
 * amplitudes of tq_amplitudes (bitstrings uint64 [B, M], amps complex64
 * [B, M], when M > 0) of the same final states.  Uses only the program's
 * cached workspaces. */
tq_status tq_sample_with_amplitudes(tq_program prog, const float *symbol_values, int64_t n_shots, uint64_t seed,
                                    uint64_t *out, const uint64_t *bitstrings, int64_t M, void *amps, void *stream);

/* Adjoint-method gradient (Sec. "Adjoint Gradient Backpropagation in
 * Simulations") of sum_k upstream[b,k] <h_{b,k}> with respect to every symbol
 * value: with H_g = sum_k g_k h_k (Sec. "Autodifferentiation through hybrid
 * quantum-classical backpropagation") it computes phi = H_g psi, then walks
 * the gates backwards, psi <- W^dagger psi, grad += scale * 2 Re <phi| dW/deta
 * |psi>, phi <- W^dagger phi.  A symbol used by several gates sums their
 * contributions (eq. chain_rule).
 * upstream: float32 [B, K]; grad: float32 [B, S] (overwritten);
 * expectations: float32 [B, K] or NULL -- when given it also receives
 * <h_{b,k}>, from the same forward pass. */
tq_status tq_adjoint_grad(tq_program prog, const float *symbol_values, tq_observables obs,
                          const float *upstream, float *grad, float *expectations, void *stream);

/* Number of non-identity terms of the row with the most (the term values
 * of tq_sampled_expectation have this many columns). */
tq_status tq_observables_terms(tq_observables obs, int32_t *Kt);

/* Expectations estimated from measurement shots (SampledExpectation; Sec.
 * "Sampling and Expectation Values": a Pauli term is measured by sampling
 * its qubits in its eigenbasis, each shot giving the parity +1 or -1).  Each
 * non-identity term t of h_{b,k} = sum_t c_t P_t is measured `reps` times on
 * its own: shot s is +1 when (u >> 11) 2^-53 < (1 + e_t) / 2, fp64, with e_t
 * the term's exact expectation as float32 clamped to [-1, 1] and u the
 * SplitMix64 output number ((b K + k) 2^40 + t 2^24 + s) of the stream
 * started at `seed` (t: the term's index in the observable, identity terms
 * counted); then out[b, k] = sum_t c_t (2 n_t / reps - 1) + the identity
 * terms' coefficients, in term order in fp64 (n_t: +1 shots), as float32.
 * The shots are drawn from exact term expectations, which gives each term's
 * shot count the distribution that sampling bitstrings would give.
 * reps in [1, 2^24); B K < 2^24; at most 65535 terms per observable
 * (TQ_E_UNSUPPORTED beyond).  out: float32 [B, K].  term_out: float32
 * [B, Kt] (tq_observables_terms) or NULL; when given it receives the term
 * expectations the shots were drawn from: row b's j-th non-identity term over
 * (k, t) in order, zero beyond the row's own. */
tq_status tq_sampled_expectation(tq_program prog, const float *symbol_values, tq_observables obs, int32_t reps,
                                 uint64_t seed, float *out, float *term_out, void *stream);

/* Gradient of sum_k upstream[b,k] <h_{b,k}> by the parameter-shift rule
 * (Sec. "Parameter shift methods", eq. parshift_grad), as batched launches:
 * every symbolic parameter of a blob gate whose generator has two
 * eigenvalues a gap r apart is moved alone by +-pi/(2r) (rotations RX, RY,
 * RZ, RZZ: +-pi/2; power gates: +-1/2 in the exponent; Pauli-string
 * exponentials: +-pi/4; fSim's phi: +-pi/2) and
 * grad[b, s] += scale x (r/2) x sum_k g_k (<h_k>(+) - <h_k>(-)) (shared
 * symbols add up, eq. chain_rule).  The shifted circuits run as derived rows
 * through the same kernels as plain rows, in chunks within fixed
 * workspaces.  reps = 0: exact expectations; reps > 0: each shifted
 * circuit's expectations are the estimates of tq_sampled_expectation, the
 * shifted circuits of all rows forming one batch of sum_b 2 O_b rows (O_b:
 * row b's symbolic parameters) in the order (row, parameter in gate and
 * parameter order, + then -), shifted circuit e taking the shot counters of
 * row e.  Noisy rows keep their trajectory.  upstream float32 [B, K], grad
 * float32 [B, S] (overwritten).  TQ_E_UNSUPPORTED for a symbolic fSim theta
 * (three generator eigenvalues: no two-term rule) or, with reps > 0, more
 * than 2^24 (shifted circuit, observable) pairs. */
tq_status tq_param_shift_grad(tq_program prog, const float *symbol_values, tq_observables obs, const float *upstream,
                              int32_t reps, uint64_t seed, float *grad, void *stream);

/* Gradient by central differences in the symbol values (Sec. "Finite
 * difference methods", eq. central_diff): grad[b, s] = sum_k g_k
 * (<h_k>(theta + eps e_s) - <h_k>(theta - eps e_s)) / (2 eps), the moved
 * symbol value formed in fp64 (theta_s + eps); symbols no gate of the row
 * uses get 0.  Batched like tq_param_shift_grad (two derived rows per symbol
 * a row uses).  eps > 0. */
tq_status tq_finite_diff_grad(tq_program prog, const float *symbol_values, tq_observables obs, const float *upstream,
                              double eps, float *grad, void *stream);

/* Amplitudes <x_{b,m}|psi_b> at M bitstrings per circuit: bitstrings uint64
 * [B, M] (each < 2^{n_b}, checked on the device: an out-of-range entry yields
 * a zero amplitude), amps complex64 [B, M]. */
tq_status tq_amplitudes(tq_program prog, const float *symbol_values, const uint64_t *bitstrings, int64_t M,
                        void *amps, void *stream);

/* The sampling rule of tq_sample applied to given states: complex64
 * [B, 2^n] device array (8-byte aligned).  Deterministic and bit-exact for a
 * given input.  Its level workspace (about B 2^n / 63 uint64) is taken from
 * the stream-ordered allocator and released in stream order on every call. */
tq_status tq_sample_from_state(const void *states, int32_t B, int32_t n, int64_t n_shots, uint64_t seed,
                               uint64_t *out, void *stream);

/* tq_sample_from_state for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same rule and kernels, bit-identical output, but no
 * allocation of any kind.  The level workspace is a static device array of
 * 2^22 uint64 (32 MiB) per GPU, held until the process ends; inputs with
 * B * (level entries per row, about 2^n / 63) above 2^22 -- e.g. B = 1 with
 * n >= 28 -- are rejected with TQ_E_UNSUPPORTED before anything is enqueued.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (other streams, other threads) race and must be serialised by the caller. */
tq_status tq_sample_from_state_noalloc(const void *states, int32_t B, int32_t n, int64_t n_shots, uint64_t seed,
                                       uint64_t *out, void *stream);

/* The amplitude lookup of tq_amplitudes applied to given states: states
 * complex64 [B, 2^n] device array, bitstrings uint64 [B, M] (an entry >= 2^n
 * yields a zero amplitude), amps complex64 [B, M].  With tq_simulate_state
 * and tq_sample_from_state it serves a state that is both sampled and
 * queried for amplitudes with one simulation. */
tq_status tq_amplitudes_from_state(const void *states, int32_t B, int32_t n, const uint64_t *bitstrings, int64_t M,
                                   void *amps, void *stream);

/* Plan introspection: a JSON description of the program's structure groups
 * and of the tile passes planned for each (tile bits, ops, fused members,
 * gradient slots).  Writes at most cap bytes (NUL terminated) into buf and
 * the full size including the NUL into *needed (either may be NULL). */
tq_status tq_program_describe(tq_program prog, char *buf, size_t cap, size_t *needed);

/* Kernel timing for benchmarks.  After tq_profile_start(name) every launch of
 * the named kernel ("build", "resident", "pass", "pauli", "pauli_reduce",
 * "rev_pass", "grad_reduce", "samp_l1", "samp_shots", "gather", "sampled_counts") is bracketed
 * by a pair of HIP events recorded on its launch stream; NULL or "" stops
 * recording.  tq_profile_read waits for the recorded events, returns the
 * number of bracketed launches and their total duration in milliseconds, and
 * clears the record.  Process-wide; not meant for concurrent use. */
tq_status tq_profile_start(const char *kernel);
tq_status tq_profile_read(int64_t *launches, double *total_ms);

/* The matrix builder's gate table, for checks on the host (no device call):
 * the matrix of opcode `op` (deriv = 0), or its derivative with respect to
 * parameter `which` (deriv = 1), at the resolved parameter values params[np],
 * as the builder forms it: without the global phase it leaves out of some
 * gates (and multiplies into the row's product state instead), which goes to
 * *phase in radians -- the gate's own matrix is e^{i phase} times `out`, and
 * the derivative is that of `out`.  explicit_m: the 8 or 32 f64 entries of
 * MATRIX1 / MATRIX2 (else NULL).  cblock = 1 asks for the 2x2 target block of
 * CNOT / CNOTPOW.  out: d*d complex128 entries, row major, interleaved
 * (re, im), host memory of at least 32 doubles; *dim = d (2 or 4).
 * TQ_E_INVALID for an unknown opcode, a null pointer, or a derivative the gate
 * does not have (gates without parameters, MATRIX1/2, SWAP). */
tq_status tq_gate_matrix(int32_t op, const double *params, const double *explicit_m, int32_t cblock, int32_t deriv,
                         int32_t which, double *out, int32_t *dim, double *phase);

/* The matrix builder's output, for checks: resolves the symbols and builds
 * every matrix of every structure group (forward products, W^dagger and
 * dW/deta of the reverse sweep, dense stage matrices) exactly as a call of
 * tq_adjoint_grad would, then copies each group's row blocks, groups in the
 * order of tq_program_describe, rows in its "row_ids" order, into out:
 * complex128 (re, im) device array of cap entries.  *entries (may be NULL)
 * receives the number of entries needed (sum over groups of rows x
 * mat_block); with out = NULL only that is returned.  The layout of a block
 * is the "tasks" list of tq_program_describe. */
tq_status tq_build_matrices(tq_program prog, const float *symbol_values, void *out, int64_t cap, int64_t *entries,
                            void *stream);

/* Message of the last failed call on this thread ("" if none). */
const char *tq_last_error(void);
const char *tq_version(void);

#ifdef __cplusplus
}
#endif
#endif /* TQ_H */
