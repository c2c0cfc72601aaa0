"""Pins of the oracle's trajectory simulation of Pauli channels (Sec. "Noise
in qsim": per trajectory one Kraus operator per channel, drawn at random;
results averaged over trajectories): the average over many trajectories
against a density-matrix simulation (oracle/dense.py), each trajectory
against the same circuit with its drawn Paulis written in as gates, the
draw frequencies against the channel's probabilities, and the edge cases."""
import math

import numpy as np
import pytest

from oracle import dense
from oracle import oracle as orc
from paper_2003_02989_amd import workloads as wl
from paper_2003_02989_amd.circuits import Circuit, const, observable_blob, program_blob, sym


def noisy_circuit(rng, n, p):
    c = Circuit(n)
    for layer in range(3):
        for q in range(n):
            c.add("RY", q, [sym(q)])
            c.depolarize(q, p)
        for q in range(n - 1):
            c.add("CNOT", (q, q + 1))
        c.add("PCHAN", int(rng.integers(0, n)), [0.05, 0.0, 0.15])
        c.add("RZ", 0, [sym(n)])
    return c


def test_trajectory_average_matches_density_matrix():
    rng = np.random.default_rng(41)
    n, R, S = 3, 4000, 4
    c = noisy_circuit(rng, n, 0.1)
    terms = [(0.8, [(0, "Z")]), (-0.5, [(1, "X"), (2, "X")]), (0.3, [(0, "Y"), (2, "Z")])]
    theta = rng.uniform(-math.pi, math.pi, size=(1, S))
    orc.set_noise_seed(1234)
    e = orc.expectation(orc.Program(program_blob([c] * R, S)), np.repeat(theta, R, 0),
                        orc.Observables(observable_blob([[terms]] * R)))[:, 0]
    want = dense.density_expectation(c.gates, n, theta[0], terms).real
    sigma = e.std() / math.sqrt(R)
    assert abs(e.mean() - want) < 4 * sigma, (e.mean(), want, sigma)
    # and the noiseless value is far outside that band (the noise matters)
    clean = Circuit(n)
    clean.gates = [g for g in c.gates if g[0] != "PCHAN"]
    assert abs(dense.expectation(clean.gates, n, theta[0], terms).real - want) > 10 * sigma


def test_each_trajectory_is_its_drawn_circuit():
    rng = np.random.default_rng(7)
    n, B, S = 4, 6, 5
    c = noisy_circuit(rng, n, 0.4)
    terms = wl.random_pauli_strings(rng, n, 5)
    theta = rng.uniform(-math.pi, math.pi, size=(B, S))
    seed = 99
    orc.set_noise_seed(seed)
    prog = orc.Program(program_blob([c] * B, S))
    st = orc.simulate_state(prog, theta)
    for b in range(B):
        explicit = Circuit(n)
        k = 0
        for name, qubits, params, matrix in c.gates:
            if name == "PCHAN":
                pk = orc.channel_pick(seed, b, k, *[off for _, _, off in params])
                k += 1
                if pk:
                    explicit.add("XYZ"[pk - 1], qubits[0])
                continue
            explicit.gates.append((name, qubits, params, matrix))
        ref = dense.state(explicit.gates, n, theta[b])
        assert np.abs(st[b] - ref).max() < 1e-12
    # the adjoint gradient of a trajectory is that of its drawn circuit
    up = np.ones((B, 1))
    g = orc.adjoint_grad(prog, theta, orc.Observables(observable_blob([[terms]] * B)), up)
    h = 1e-6
    # central differences of the trajectory itself (same rows, same draws)
    for s in range(S):
        tp, tm = theta.copy(), theta.copy()
        tp[:, s] += h
        tm[:, s] -= h
        o = orc.Observables(observable_blob([[terms]] * B))
        fd = (orc.expectation(prog, tp, o) - orc.expectation(prog, tm, o))[:, 0] / (2 * h)
        assert np.abs(g[:, s] - fd).max() < 1e-7


def test_draw_frequencies():
    # 200000 draws of one channel against its probabilities (chi-squared,
    # 3 degrees of freedom, p-value far below 1e-6 excluded)
    p = (0.1, 0.25, 0.05)
    counts = np.zeros(4)
    for row in range(200_000):
        counts[orc.channel_pick(5, row, 3, *p)] += 1
    probs = np.array([1 - sum(p), *p])
    chi2 = (((counts - 2e5 * probs) ** 2) / (2e5 * probs)).sum()
    assert chi2 < 35.0, (counts, chi2)
    # edge cases: p = 0 never fires, probabilities summing to 1 never give I
    assert all(orc.channel_pick(1, r, 0, 0.0, 0.0, 0.0) == 0 for r in range(2000))
    assert all(orc.channel_pick(1, r, 0, 0.5, 0.0, 0.5) in (1, 3) for r in range(2000))


def test_seeds_and_rejects():
    rng = np.random.default_rng(3)
    c = noisy_circuit(rng, 3, 0.5)
    theta = rng.uniform(-1, 1, size=(4, 4))
    prog = orc.Program(program_blob([c] * 4, 4))
    orc.set_noise_seed(1)
    a = orc.simulate_state(prog, theta)
    orc.set_noise_seed(1)
    assert np.array_equal(a, orc.simulate_state(prog, theta))
    orc.set_noise_seed(2)
    assert not np.array_equal(a, orc.simulate_state(prog, theta))
    # a channel with zero probabilities is the noiseless circuit
    z = Circuit(2).add("H", 0).add("PCHAN", 0, [0.0, 0.0, 0.0]).add("CNOT", (0, 1))
    st = orc.simulate_state(orc.Program(program_blob([z], 0)), np.zeros((1, 0)))
    assert np.allclose(st[0], [2 ** -0.5, 0, 0, 2 ** -0.5], atol=1e-15)
    for params in ([0.5, 0.6, 0.0], [-0.1, 0.0, 0.0], [sym(0), 0.0, 0.0]):
        bad = Circuit(2).add("PCHAN", 0, params)
        with pytest.raises(Exception):
            orc.Program(program_blob([bad], 1))
