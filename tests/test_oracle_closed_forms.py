"""Pins of the oracle against closed forms: the worked examples the paper
prints, textbook states (Bell, GHZ, cluster) and the special cases of the
five workload configurations that reduce to a product state."""
import math

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2003_02989_amd import workloads as wl
from paper_2003_02989_amd.circuits import Circuit, const, observable_blob, program_blob, sym


def run(circuits, S, theta, obs):
    p = orc.Program(program_blob(circuits, S))
    o = orc.Observables(observable_blob(obs))
    return orc.expectation(p, theta, o, return_imag=True)


def test_bell_zz_and_amplitudes():
    # Sec. "Cirq": H then CNOT, <Z1 Z2> of the Bell state
    c = Circuit(2).add("H", 0).add("CNOT", (0, 1))
    e, im = run([c], 0, np.zeros((1, 0)), [[[(1.0, [(0, "Z"), (1, "Z")])]]])
    assert abs(e[0, 0] - 1.0) < 1e-14 and abs(im[0, 0]) < 1e-14
    st = orc.simulate_state(orc.Program(program_blob([c], 0)), np.zeros((1, 0)))
    r = 1 / math.sqrt(2)
    assert np.allclose(st[0], [r, 0, 0, r], atol=1e-15)


def test_x_power_theta_batch():
    # Sec. "Design Principles and Overview": X**theta on |0>, theta in {0,1,2}, <Z>
    c = Circuit(1).add("XPOW", 0, [sym(0)])
    e, _ = run([c] * 3, 1, np.array([[0.0], [1.0], [2.0]]), [[[(1.0, [(0, "Z")])]]] * 3)
    assert np.allclose(e[:, 0], [1.0, -1.0, 1.0], atol=1e-14)


def test_ry_after_h_half_z():
    # Sec. "Quantum Computations as Tensors": H, then Ry(theta), theta=0.5, observable 0.5 Z
    c = Circuit(1).add("H", 0).add("RY", 0, [sym(0)])
    e, _ = run([c], 1, np.array([[0.5]]), [[[(0.5, [(0, "Z")])]]])
    assert abs(e[0, 0] - (-0.5 * math.sin(0.5))) < 1e-15
    assert abs(e[0, 0] - (-0.2397128)) < 1e-7


def test_pqc_and_controlled_pqc_rows():
    # Sec. "Simplified Layers": Rz(a) Rx(b) appended to the empty circuit and to X|0>
    def model(data_x):
        c = Circuit(1)
        if data_x:
            c.add("X", 0)
        c.add("RZ", 0, [sym(0)]).add("RX", 0, [sym(1)])
        return c
    th = np.array([[0.5, 0.5], [0.25, 0.75]])
    e, _ = run([model(False), model(True)], 2, th, [[[(1.0, [(0, "Z")])]]] * 2)
    assert np.allclose(e[:, 0], [math.cos(0.5), -math.cos(0.75)], atol=1e-15)
    assert abs(e[0, 0] - 0.8775826) < 1e-7 and abs(e[1, 0] + 0.7316889) < 1e-7


@pytest.mark.parametrize("phi", [0.0, 0.4, 2.0, -1.3])
def test_h_rz_x_expectation(phi):
    # Sec. "Time-dependent Hamiltonian Control": H then Rz(phi), <X> = cos(phi)
    c = Circuit(1).add("H", 0).add("RZ", 0, [sym(0)])
    e, _ = run([c], 1, np.array([[phi]]), [[[(1.0, [(0, "X")])]]])
    assert abs(e[0, 0] - math.cos(phi)) < 1e-14


@pytest.mark.parametrize("theta", np.linspace(-3, 6, 7))
def test_rx_z(theta):
    c = Circuit(1).add("RX", 0, [sym(0)])
    e, _ = run([c], 1, np.array([[theta]]), [[[(1.0, [(0, "Z")])]]])
    assert abs(e[0, 0] - math.cos(theta)) < 1e-14


@pytest.mark.parametrize("n", [3, 5, 8])
def test_cluster_state_stabilizers(n):
    # Sec. "Hybrid Quantum-Classical Convolutional Neural Network Classifier":
    # H on all qubits then CZ on the ring; Z_{i-1} X_i Z_{i+1} stabilizes it
    c = Circuit(n)
    for q in range(n):
        c.add("H", q)
    for q in range(n):
        c.add("CZ", (q, (q + 1) % n))
    obs = [[(1.0, [((i - 1) % n, "Z"), (i, "X"), ((i + 1) % n, "Z")])] for i in range(n)]
    obs += [[(1.0, [(i, "X")])] for i in range(n)]
    e, im = run([c], 0, np.zeros((1, 0)), [obs])
    assert np.allclose(e[0, :n], 1.0, atol=1e-13)
    assert np.allclose(e[0, n:], 0.0, atol=1e-13)
    assert np.abs(im).max() < 1e-13


@pytest.mark.parametrize("n", [2, 4, 7])
def test_ghz(n):
    c = Circuit(n).add("H", 0)
    for q in range(n - 1):
        c.add("CNOT", (q, q + 1))
    st = orc.simulate_state(orc.Program(program_blob([c], 0)), np.zeros((1, 0)))[0]
    ref = np.zeros(1 << n, complex)
    ref[0] = ref[-1] = 1 / math.sqrt(2)
    assert np.abs(st - ref).max() < 1e-15
    obs = [[(1.0, [(0, "Z"), (n - 1, "Z")])], [(1.0, [(q, "X") for q in range(n)])]]
    e, _ = run([c], 0, np.zeros((1, 0)), [obs])
    assert np.allclose(e[0], [1.0, 1.0], atol=1e-14)


def _oracle_of(w):
    return orc.Program(w.program_blob()), orc.Observables(w.observable_blob())


def test_c1_zero_angles():
    w = wl.c1_hea(B=2)
    p, o = _oracle_of(w)
    e = orc.expectation(p, np.zeros((2, w.n_symbols)), o)
    assert np.allclose(e, 4.0, atol=1e-14)


def test_c2_zero_angles():
    w = wl.c2_qnn(B=4)
    p, o = _oracle_of(w)
    e = orc.expectation(p, np.zeros((4, w.n_symbols)), o)
    assert np.allclose(e, 1.0, atol=1e-14)


def test_c3_zero_gamma():
    # gamma = 0: the cost layers vanish, H^n|0> = |+>^n is an eigenstate of
    # every RX, so <C> = |E|/2 = 15 for any beta, and d<C>/d beta = 0
    w = wl.c3_qaoa(B=3, n=8)
    th = w.theta.astype(np.float64).copy()
    th[:, :4] = 0
    p, o = _oracle_of(w)
    e = orc.expectation(p, th, o)
    assert np.allclose(e, len(w.extras["edges"]) / 2, atol=1e-13)
    g = orc.adjoint_grad(p, th, o, np.ones((3, 1)))
    assert np.abs(g[:, 4:]).max() < 1e-13


def test_c5_zero_angles():
    # theta = 0: the ansatz leaves |0..0> (CNOTs act trivially), so <H> is the
    # sum of the coefficients of the Z-only strings
    w = wl.c5_vqe(B=2, n=8, layers=2, n_terms=40)
    p, o = _oracle_of(w)
    e = orc.expectation(p, np.zeros((2, w.n_symbols)), o)
    want = sum(c for c, f in w.observables[0][0] if all(pq == "Z" for _, pq in f))
    assert np.allclose(e, want, atol=1e-13)


def test_identity_term_and_empty_circuit():
    c = Circuit(3)
    e, _ = run([c], 0, np.zeros((1, 0)), [[[(2.5, []), (1.0, [(2, "Z")]), (1.0, [(1, "X")])]]])
    assert abs(e[0, 0] - 3.5) < 1e-15


@pytest.mark.parametrize("seed", range(3))
def test_product_state_pauli_strings(seed):
    # RY(t) then RZ(f) on every qubit: a product state whose Bloch vectors are
    # (sin t cos f, sin t sin f, cos t); a Pauli string's expectation is its
    # coefficient times the product of its factors' components (X/Y/Z strings
    # of any weight, several observables, identity terms)
    rng = np.random.default_rng(70 + seed)
    n, B = 6, 3
    c = Circuit(n)
    for q in range(n):
        c.add("RY", q, [sym(q)]).add("RZ", q, [sym(n + q)])
    obs = [wl.random_pauli_strings(rng, n, 25, max_weight=n) + [(0.3, [])] for _ in range(3)]
    theta = rng.uniform(0.0, 2 * math.pi, size=(B, 2 * n))
    e, im = run([c] * B, 2 * n, theta, [obs] * B)
    for b in range(B):
        t, f = theta[b, :n], theta[b, n:]
        comp = [{"X": math.sin(t[q]) * math.cos(f[q]), "Y": math.sin(t[q]) * math.sin(f[q]), "Z": math.cos(t[q])}
                for q in range(n)]
        for k, terms in enumerate(obs):
            ref = sum(cf * np.prod([comp[q][p] for q, p in fac]) for cf, fac in terms)
            assert abs(e[b, k] - ref) < 1e-13 and abs(im[b, k]) < 1e-13
