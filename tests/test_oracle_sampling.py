"""Pins of the oracle's sampler: a chi-squared goodness-of-fit test against
|psi_i|^2, degenerate states, zero-probability outcomes, the counter
stream's published values, and the Bell state of Sec. "Cirq"."""
import math

import numpy as np
from scipy import stats

from oracle import oracle as orc
from paper_2003_02989_amd.circuits import Circuit, program_blob


def test_chi_squared_fit():
    rng = np.random.default_rng(3)
    for n in (3, 6, 10):
        N = 1 << n
        z = (rng.standard_normal(N) + 1j * rng.standard_normal(N)).astype(np.complex64)
        z /= np.linalg.norm(z)
        shots = 200_000
        s = orc.sample_from_state(z[None, :], shots, seed=11)[0]
        counts = np.bincount(s.astype(np.int64), minlength=N)
        p = np.abs(z.astype(np.complex128)) ** 2
        p /= p.sum()
        chi2 = ((counts - shots * p) ** 2 / (shots * p)).sum()
        assert stats.chi2.sf(chi2, N - 1) > 1e-4, n


def test_basis_state_and_zero_weights():
    N = 16
    z = np.zeros((1, N), np.complex64)
    z[0, 9] = 1j
    s = orc.sample_from_state(z, 1000, seed=5)
    assert np.all(s == 9)
    z = np.zeros((1, N), np.complex64)
    z[0, [2, 7, 13]] = [0.6, 0.0, 0.8j]
    s = orc.sample_from_state(z, 5000, seed=1)
    assert set(np.unique(s).tolist()) == {2, 13}


def test_bell_state_samples():
    c = Circuit(2).add("H", 0).add("CNOT", (0, 1))
    s = orc.sample(orc.Program(program_blob([c], 0)), np.zeros((1, 0)), 20_000, seed=123)[0]
    assert set(np.unique(s).tolist()) == {0, 3}
    frac = (s == 3).mean()
    assert abs(frac - 0.5) < 5 * math.sqrt(0.25 / 20_000)


def test_rows_use_distinct_counters_and_seed_changes_stream():
    z = np.full((2, 64), 1 / 8, np.complex64)
    a = orc.sample_from_state(z, 100, seed=9)
    assert not np.array_equal(a[0], a[1])
    b = orc.sample_from_state(z, 100, seed=10)
    assert not np.array_equal(a, b)
    assert np.array_equal(a, orc.sample_from_state(z, 100, seed=9))


def test_zero_row_gives_the_marker():
    # a row with no weight has no distribution: every shot is 2^64 - 1 (no
    # bitstring of at most 34 qubits), and the other rows draw as usual
    z = np.zeros((3, 32), np.complex64)
    z[0, 5] = 1.0
    z[2, [1, 30]] = [0.6, 0.8]
    s = orc.sample_from_state(z, 400, seed=17)
    assert np.all(s[1] == np.uint64(2**64 - 1))
    assert np.all(s[0] == 5)
    assert set(np.unique(s[2]).tolist()) <= {1, 30}
    alone = orc.sample_from_state(z[2:], 400, seed=17)
    # row 2 of the batch uses counters 2 * 400 + k, row 0 of `alone` 0 * 400 + k
    assert alone.shape == (1, 400)
