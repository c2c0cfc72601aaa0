"""Pin of the oracle's simulator against dense brute force: random circuits
over the whole opcode set on n <= 5 qubits, compared with the product of
full 2^n x 2^n unitaries built from the gates' generators (oracle/dense.py)."""
import numpy as np
import pytest

from oracle import dense
from oracle import oracle as orc
from paper_2003_02989_amd import workloads as wl


@pytest.mark.parametrize("seed", range(6))
def test_random_circuits_against_dense(seed):
    w = wl.random_batch(1000 + seed, B=4, n=5, n_gates=30, n_symbols=4, K=3, hetero=True)
    prog = orc.Program(w.program_blob())
    obs = orc.Observables(w.observable_blob())
    th = w.theta.astype(np.float64)
    st = orc.simulate_state(prog, th)
    e, im = orc.expectation(prog, th, obs, return_imag=True)
    for b, c in enumerate(w.circuits):
        ref = dense.state(c.gates, c.n, th[b])
        N = 1 << c.n
        assert np.abs(st[b, :N] - ref).max() < 1e-12
        assert not np.any(st[b, N:])  # zero padding beyond 2^n_b
        assert abs(np.linalg.norm(st[b]) - 1) < 1e-12
        for k in range(w.K):
            want = dense.expectation(c.gates, c.n, th[b], w.observables[b][k])
            assert abs(e[b, k] - want.real) < 1e-12
            assert abs(want.imag) < 1e-12 and abs(im[b, k]) < 1e-12


def test_amplitudes_match_state():
    w = wl.random_batch(77, B=3, n=5, n_gates=25, n_symbols=2, K=1)
    prog = orc.Program(w.program_blob())
    th = w.theta.astype(np.float64)
    st = orc.simulate_state(prog, th)
    bits = np.random.default_rng(1).integers(0, 32, size=(3, 9)).astype(np.uint64)
    a = orc.amplitudes(prog, th, bits)
    for b in range(3):
        assert np.array_equal(a[b], st[b, bits[b].astype(np.int64)])


def test_bitstring_convention():
    # qubit 0 is the most significant bit: X on qubit 0 of 3 gives index 4
    from paper_2003_02989_amd.circuits import Circuit, program_blob
    c = Circuit(3).add("X", 0)
    st = orc.simulate_state(orc.Program(program_blob([c], 0)), np.zeros((1, 0)))
    assert st[0, 4] == 1 and np.abs(st[0]).sum() == 1
