"""Program and observable blobs: the wire format of the tq C-ABI.

A circuit batch is data, not code (the paper serializes Cirq circuits and
Pauli sums into string tensors so that a new circuit needs no graph rebuild,
Sec. "TFQ architecture" and "Quantum Computations as Tensors").  Here the
serialization is a flat little-endian blob that ``tq_program_create`` and
``tq_observables_create`` parse.  This module only writes bytes: it holds no
simulation arithmetic.

Program blob::

    "TQP1" u32 version=1  u32 B  u32 S
    per circuit:  u32 n_qubits  u32 n_gates
      per gate:   u16 opcode  u8 nq  u8 np  u32 qubit[nq]
                  np x { i32 symbol (-1 = constant)  f64 scale  f64 offset }
                  MATRIX1: 8 f64, MATRIX2: 32 f64 (re, im interleaved, row major)
                  PAULIEXP: nq u8 Pauli codes (1=X 2=Y 3=Z), one per qubit

PCHAN (opcode 27) is a Pauli channel on one qubit: X, Y or Z with the
constant probabilities (p_x, p_y, p_z) of its three parameters, else the
identity.  Noisy circuits run as trajectories (Sec. "Noise in qsim"): every
batch row draws one Pauli per channel from a counter stream seeded per call,
so R rows holding the same circuit are R trajectories of it.

PAULIEXP (opcode 26) is exp(-i eta P) for the Pauli string P over its nq
qubits (any weight, nq = 0 being a global phase), the exponentials of the
Pauli decomposition of a generator (Sec. "Quantum Neural Networks",
eqs. Pauli_decomp and cs_decomp) that the paper's exponential utility builds
from a Pauli sum term by term.

Each parameter resolves to eta = scale * symbol_values[b, symbol] + offset
(or eta = offset for a constant), the affine symbol expressions of the
paper's chain rule (Sec. "Parameter shift methods", eq. chain_rule).

Observable blob::

    "TQO1" u32 version=1  u32 B  u32 K
    per (b, k), row major:  u32 T
      per term:  f64 coeff  u32 n_factors  n_factors x { u32 qubit  u8 pauli (1=X 2=Y 3=Z) }

An empty factor list is the identity term.

Qubit q of an n-qubit circuit is bit (n-1-q) of an amplitude index and of a
sampled bitstring; a two-qubit gate on (a, b) has local index 2*bit(a)+bit(b).
"""
import struct

import numpy as np

# name -> (opcode, n_qubits, n_params)
OPS = {
    "H": (1, 1, 0), "X": (2, 1, 0), "Y": (3, 1, 0), "Z": (4, 1, 0),
    "RX": (5, 1, 1), "RY": (6, 1, 1), "RZ": (7, 1, 1),
    "XPOW": (8, 1, 1), "YPOW": (9, 1, 1), "ZPOW": (10, 1, 1),
    "CZ": (11, 2, 0), "CNOT": (12, 2, 0), "CZPOW": (13, 2, 1), "CNOTPOW": (14, 2, 1),
    "XXPOW": (15, 2, 1), "YYPOW": (16, 2, 1), "ZZPOW": (17, 2, 1), "RZZ": (18, 2, 1),
    "SQRTX": (19, 1, 0), "SQRTY": (20, 1, 0), "SQRTW": (21, 1, 0),
    "FSIM": (22, 2, 2), "MATRIX1": (23, 1, 0), "MATRIX2": (24, 2, 0), "SWAP": (25, 2, 0),
    "PAULIEXP": (26, None, 1),
    "PCHAN": (27, 1, 3),
}
OPCODE_NAMES = {v[0]: k for k, v in OPS.items()}
PAULI_CODES = {"X": 1, "Y": 2, "Z": 3}


def sym(index, scale=1.0, offset=0.0):
    """A symbolic parameter: eta = scale * symbol_values[b, index] + offset."""
    return (int(index), float(scale), float(offset))


def const(value):
    """A constant parameter."""
    return (-1, 0.0, float(value))


class Circuit:
    """An n-qubit gate list.  Parameters are (symbol, scale, offset) triples
    (see ``sym`` / ``const``) or plain numbers (constants)."""

    def __init__(self, n_qubits):
        self.n = int(n_qubits)
        self.gates = []

    def add_pauli_exp(self, factors, param):
        """exp(-i eta P) for the Pauli string ``factors`` = [(qubit, 'X'|'Y'|'Z'), ...]
        (distinct qubits; an empty list is the global phase exp(-i eta)); the
        string's letters ride in the gate's matrix slot."""
        qubits = tuple(int(q) for q, _ in factors)
        letters = "".join(p for _, p in factors)
        if any(p not in PAULI_CODES for p in letters):
            raise ValueError("Pauli factors are X, Y or Z")
        self.gates.append(("PAULIEXP", qubits, (param if isinstance(param, tuple) else const(param),), letters))
        return self

    def depolarize(self, qubit, p):
        """Depolarizing channel: X, Y or Z each with probability p / 3."""
        return self.add("PCHAN", qubit, [p / 3.0, p / 3.0, p / 3.0])

    def bit_flip(self, qubit, p):
        return self.add("PCHAN", qubit, [p, 0.0, 0.0])

    def phase_flip(self, qubit, p):
        return self.add("PCHAN", qubit, [0.0, 0.0, p])

    def add(self, name, qubits, params=(), matrix=None):
        code, nq, npar = OPS[name]
        if nq is None:
            raise ValueError(f"{name} is added with add_pauli_exp")
        qubits = tuple(int(q) for q in (qubits if isinstance(qubits, (tuple, list)) else (qubits,)))
        if len(qubits) != nq:
            raise ValueError(f"{name} takes {nq} qubits")
        ps = []
        for p in params:
            ps.append(p if isinstance(p, tuple) else const(p))
        if len(ps) != npar:
            raise ValueError(f"{name} takes {npar} parameters")
        self.gates.append((name, qubits, tuple(ps), None if matrix is None else np.asarray(matrix, np.complex128)))
        return self

    def __len__(self):
        return len(self.gates)


def _circuit_bytes(c):
    out = [struct.pack("<II", c.n, len(c.gates))]
    for name, qubits, params, matrix in c.gates:
        code, nq, npar = OPS[name]
        nq = len(qubits)
        out.append(struct.pack("<HBB", code, nq, npar))
        out.append(struct.pack(f"<{nq}I", *qubits))
        for s, scale, offset in params:
            out.append(struct.pack("<idd", s, scale, offset))
        if name == "PAULIEXP":
            out.append(bytes(PAULI_CODES[p] for p in matrix))
        if name in ("MATRIX1", "MATRIX2"):
            d = 2 if name == "MATRIX1" else 4
            m = np.asarray(matrix, np.complex128).reshape(d, d)
            out.append(np.stack([m.real.ravel(), m.imag.ravel()], axis=1).astype("<f8").tobytes())
    return b"".join(out)


def program_blob(circuits, n_symbols):
    # a circuit object repeated in the batch (trajectories, uniform batches)
    # is encoded once
    memo = {}
    out = [b"TQP1", struct.pack("<III", 1, len(circuits), int(n_symbols))]
    for c in circuits:
        b = memo.get(id(c))
        if b is None:
            b = memo[id(c)] = _circuit_bytes(c)
        out.append(b)
    return b"".join(out)


def observable_blob(sums):
    """``sums[b][k]`` is a list of terms ``(coeff, [(qubit, 'X'|'Y'|'Z'), ...])``."""
    B = len(sums)
    K = len(sums[0]) if B else 0
    out = [b"TQO1", struct.pack("<III", 1, B, K)]
    memo = {}  # a row object repeated in the batch is encoded once
    for row in sums:
        if len(row) != K:
            raise ValueError("every batch row needs the same number of observables")
        b = memo.get(id(row))
        if b is None:
            enc = []
            for terms in row:
                enc.append(struct.pack("<I", len(terms)))
                for coeff, factors in terms:
                    enc.append(struct.pack("<dI", float(coeff), len(factors)))
                    for q, p in factors:
                        enc.append(struct.pack("<IB", int(q), PAULI_CODES[p]))
            b = memo[id(row)] = b"".join(enc)
        out.append(b)
    return b"".join(out)
