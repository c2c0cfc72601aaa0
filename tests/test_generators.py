"""Gate generators used by the specialised reverse kernels (CPU only).

The generated reverse stages take the gradient of a parameter eta of a gate
W(eta) = exp(-i eta G) (times factors commuting with G) as Im<phi|G|psi>
on the state after the gate, where the table-driven kernels multiply by
dW/deta: the two agree when G = i (dW/deta) W^dagger for every eta.  The
planner's generator terms (exported per reverse op in the plan description)
are checked here against that product, formed from the oracle's own gate
matrices and derivatives at random parameter values (Sec. "Adjoint Gradient
Backpropagation in Simulations").
"""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_2003_02989_amd import tq
from paper_2003_02989_amd.circuits import OPS, Circuit, program_blob, sym

PARAM_GATES = sorted(name for name, (_, nq, npar) in OPS.items() if npar > 0 and nq is not None and name != "PCHAN")

X = np.array([[0, 1], [1, 0]], dtype=complex)
Z = np.diag([1.0, -1.0]).astype(complex)
I2 = np.eye(2, dtype=complex)


def pauli_term_matrix(x, z, ny, nq, q0_weight, q1_weight):
    """i^ny X^x Z^z on the op's qubits (bit 0: q0, bit 1: q1) as a matrix
    over the gate's local index, where q0 / q1 carry the given bit weights."""
    d = 1 << nq
    m = np.zeros((d, d), dtype=complex)
    for col in range(d):
        # op-frame bits of the basis state |col>
        b0 = (col // q0_weight) & 1
        b1 = (col // q1_weight) & 1 if nq == 2 else 0
        # Z^z then X^x: sign from the bits of col, then flip the x bits
        sign = (-1) ** (((z & 1) and b0) + ((z & 2 and nq == 2) and b1))
        row = col
        if x & 1:
            row ^= q0_weight
        if x & 2:
            row ^= q1_weight
        m[row, col] += (1j ** ny) * sign
    return m


def single_gate_plan(name, qubits, n=3):
    _, nq, npar = OPS[name]
    c = Circuit(n)
    c.add(name, qubits, [sym(j, 1.0, 0.0) for j in range(npar)])
    p = tq.Program(program_blob([c], npar))
    plan = tq.describe(p)
    rev_ops = [op for ps in plan["groups"][0]["rev"] for op in ps["ops"]]
    assert len(rev_ops) == 1
    return rev_ops[0]


@pytest.mark.parametrize("name", PARAM_GATES)
def test_generator_terms_match_oracle_derivatives(name):
    opcode, nq, npar = OPS[name]
    qubits = (1,) if nq == 1 else (2, 0)
    op = single_gate_plan(name, qubits)
    assert op["ngrad"] == npar and len(op["gen"]) == npar
    # op frame: a controlled gate's op acts on (target, control); in the
    # gate's local index the first qubit has weight 2, the second weight 1
    if nq == 1:
        w0, w1 = 1, 0
    elif op["ctrl"]:
        w0, w1 = 1, 2
    else:
        w0, w1 = 2, 1
    rng = np.random.default_rng(opcode)
    for _ in range(3):
        params = rng.uniform(-np.pi, np.pi, size=npar)
        W = orc.gate_matrix(opcode, params)
        for j in range(npar):
            terms = op["gen"][j]
            assert terms, f"{name}: no generator for parameter {j}"
            G = sum(c * pauli_term_matrix(x, z, ny, nq, w0, w1) for x, z, ny, c in terms)
            dW = orc.gate_dmatrix(opcode, params, j)
            np.testing.assert_allclose(G, 1j * dW @ W.conj().T, atol=1e-12, err_msg=f"{name} param {j}")
            np.testing.assert_allclose(G, G.conj().T, atol=1e-15)


def test_constant_gates_have_no_gradient_terms():
    c = Circuit(2)
    c.add("H", (0,), [])
    c.add("CNOT", (0, 1), [])
    c.add("RX", (1,), [(-1, 0.0, 0.3)])
    plan = tq.describe(tq.Program(program_blob([c], 1)))
    for ps in plan["groups"][0]["rev"]:
        for op in ps["ops"]:
            assert op["ngrad"] == 0 and op["gen"] == []
