"""Dense brute force for tiny circuits (n <= 6): the oracle's own cross-check.

TEST INFRASTRUCTURE ONLY.  Independent of tq_oracle.c: every gate is built
here from its generator with a matrix exponential (a rotation is
exp(-i theta G / 2), a power gate is G^t = exp(i pi t (I - G) / 2), fSim is
exp(-i theta (XX + YY) / 2) times a controlled phase, a Pauli-string
exponential is exp(-i eta P)), embedded in the full
2^n x 2^n space by index arithmetic, and the circuit unitary is the plain
matrix product (Sec. "Quantum Neural Networks", eq. full_par_circ).  Pauli
sums are Kronecker products of 2x2 Paulis (eq. cost_lincomb).

Input is the plain gate list ``[(name, qubits, params, matrix)]`` where each
param is (symbol, scale, offset), as held by ``Circuit.gates``.
"""
import numpy as np
from scipy.linalg import expm

I2 = np.eye(2, dtype=complex)
PX = np.array([[0, 1], [1, 0]], dtype=complex)
PY = np.array([[0, -1j], [1j, 0]], dtype=complex)
PZ = np.array([[1, 0], [0, -1]], dtype=complex)
PAULI = {"X": PX, "Y": PY, "Z": PZ}


def _pow(G, t):
    d = G.shape[0]
    return expm(1j * np.pi * t / 2 * (np.eye(d) - G))


def _rot(G, theta):
    return expm(-1j * theta / 2 * G)


def gate(name, eta=(), matrix=None):
    XX, YY, ZZ = np.kron(PX, PX), np.kron(PY, PY), np.kron(PZ, PZ)
    CZ = np.diag([1, 1, 1, -1]).astype(complex)
    CNOT = np.kron(np.diag([1, 0]), I2) + np.kron(np.diag([0, 1]), PX)
    W = (PX + PY) / np.sqrt(2)
    if name == "H":
        return (PX + PZ) / np.sqrt(2)
    if name in ("X", "Y", "Z"):
        return PAULI[name].copy()
    if name in ("RX", "RY", "RZ"):
        return _rot(PAULI[name[1]], eta[0])
    if name in ("XPOW", "YPOW", "ZPOW"):
        return _pow(PAULI[name[0]], eta[0])
    if name == "SQRTX":
        return _pow(PX, 0.5)
    if name == "SQRTY":
        return _pow(PY, 0.5)
    if name == "SQRTW":
        return _pow(W, 0.5)
    if name == "CZ":
        return CZ
    if name == "CNOT":
        return CNOT
    if name == "SWAP":
        return (np.eye(4) + XX + YY + ZZ).astype(complex) / 2
    if name == "CZPOW":
        return _pow(CZ, eta[0])
    if name == "CNOTPOW":
        return _pow(CNOT, eta[0])
    if name == "XXPOW":
        return _pow(XX, eta[0])
    if name == "YYPOW":
        return _pow(YY, eta[0])
    if name == "ZZPOW":
        return _pow(ZZ, eta[0])
    if name == "RZZ":
        return _rot(ZZ, eta[0])
    if name == "FSIM":
        return expm(-1j * eta[0] / 2 * (XX + YY)) @ np.diag([1, 1, 1, np.exp(-1j * eta[1])])
    if name in ("MATRIX1", "MATRIX2"):
        return np.asarray(matrix, dtype=complex)
    if name == "PAULIEXP":  # the letters of the string ride in the matrix slot
        P = np.array([[1.0 + 0j]])
        for p in matrix:
            P = np.kron(P, PAULI[p])
        return expm(-1j * eta[0] * P)
    raise ValueError(name)


def embed(M, qubits, n):
    """Full-space operator of M acting on `qubits` (first qubit = most
    significant local bit); qubit q is bit n-1-q of the global index."""
    N = 1 << n
    idx = np.arange(N)
    k = len(qubits)
    loc = np.zeros(N, dtype=np.int64)
    mask = 0
    for j, q in enumerate(qubits):
        loc |= ((idx >> (n - 1 - q)) & 1) << (k - 1 - j)
        mask |= 1 << (n - 1 - q)
    rest = idx & ~mask
    return M[loc[:, None], loc[None, :]] * (rest[:, None] == rest[None, :])


def resolve(params, theta_row):
    return [scale * float(theta_row[s]) + offset if s >= 0 else offset for s, scale, offset in params]


def unitary(gates, n, theta_row):
    U = np.eye(1 << n, dtype=complex)
    for name, qubits, params, matrix in gates:
        U = embed(gate(name, resolve(params, theta_row), matrix), qubits, n) @ U
    return U


def state(gates, n, theta_row):
    return unitary(gates, n, theta_row)[:, 0]


def pauli_sum(terms, n):
    H = np.zeros((1 << n, 1 << n), dtype=complex)
    for coeff, factors in terms:
        ops = [I2] * n
        for q, p in factors:
            ops[q] = PAULI[p]
        P = np.array([[1.0 + 0j]])
        for o in ops:
            P = np.kron(P, o)
        H += coeff * P
    return H


def expectation(gates, n, theta_row, terms):
    psi = state(gates, n, theta_row)
    return np.vdot(psi, pauli_sum(terms, n) @ psi)


def density_expectation(gates, n, theta_row, terms):
    """tr(H rho) with rho evolved as a density matrix: unitaries as U rho U^dag,
    a Pauli channel (p_x, p_y, p_z) as (1 - p) rho + sum_k p_k P_k rho P_k
    (Sec. "Noise in qsim", the full-density-matrix alternative to trajectories)."""
    N = 1 << n
    rho = np.zeros((N, N), dtype=complex)
    rho[0, 0] = 1.0
    for name, qubits, params, matrix in gates:
        eta = resolve(params, theta_row)
        if name == "PCHAN":
            out = (1.0 - sum(eta)) * rho
            for p, P in zip(eta, (PX, PY, PZ)):
                E = embed(P, qubits, n)
                out = out + p * (E @ rho @ E.conj().T)
            rho = out
            continue
        U = embed(gate(name, eta, matrix), qubits, n)
        rho = U @ rho @ U.conj().T
    return np.trace(pauli_sum(terms, n) @ rho)
