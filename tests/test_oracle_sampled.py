"""Pins of the oracle's sampled expectation (Sec. "Sampling and Expectation
Values": expectations as averages over measurement shots): each
non-identity term measured `reps` times, a shot +1 with probability
(1 + <P>)/2.  Checked against the exact expectation within the binomial
standard error, exactly on eigenstates and identity terms, the shot count's
mean and variance against the binomial law, and the estimate from given term
values against the full pipeline."""
import math

import numpy as np

from oracle import oracle as orc
from paper_2003_02989_amd import workloads as wl
from paper_2003_02989_amd.circuits import Circuit, const, observable_blob, program_blob


def test_estimate_within_binomial_error():
    w = wl.random_batch(610, B=3, n=5, n_gates=30, n_symbols=3, K=2)
    prog = orc.Program(w.program_blob())
    obs = orc.Observables(w.observable_blob())
    th = w.theta.astype(np.float64)
    exact = orc.expectation(prog, th, obs)
    reps = 20000
    est = orc.sampled_expectation(prog, th, obs, reps, 5)
    for b in range(w.B):
        for k in range(w.K):
            var = 0.0
            for c, fac in w.observables[b][k]:
                if fac:
                    e = orc.expectation(prog, th, orc.Observables(observable_blob([[[(1.0, fac)]] * 1] * w.B)))[b, 0]
                    var += c * c * (1 - e * e) / reps
            assert abs(est[b, k] - exact[b, k]) <= 5 * math.sqrt(var) + 1e-12, (b, k, est[b, k], exact[b, k], var)


def test_eigenstates_and_identity_terms_are_exact():
    # |0..0> after X on qubit 1: Z_0 = +1, Z_1 = -1 exactly; identity terms
    # carry their coefficient; X_0 has <X> = 0 (sampled)
    c = Circuit(3).add("X", 1)
    prog = orc.Program(program_blob([c], 0))
    obs = orc.Observables(observable_blob([[[(0.5, [(0, "Z")]), (-2.0, [(1, "Z")]), (1.25, [])], [(3.0, [])]]]))
    est = orc.sampled_expectation(prog, np.zeros((1, 0)), obs, 100, 1)
    assert est[0, 0] == 0.5 + 2.0 + 1.25 and est[0, 1] == 3.0


def test_shot_counts_follow_the_binomial_law():
    # RY(t)|0>: <Z> = cos t; over 400 seeds the estimate of Z (reps = 50) has
    # mean cos t and variance (1 - cos^2 t) / 50
    t = 1.1
    c = Circuit(1).add("RY", 0, [const(t)])
    prog = orc.Program(program_blob([c], 0))
    obs = orc.Observables(observable_blob([[[(1.0, [(0, "Z")])]]]))
    reps, runs = 50, 400
    x = np.array([orc.sampled_expectation(prog, np.zeros((1, 0)), obs, reps, s)[0, 0] for s in range(runs)])
    mu, var = math.cos(t), (1 - math.cos(t) ** 2) / reps
    assert abs(x.mean() - mu) < 5 * math.sqrt(var / runs)
    assert abs(x.var() / var - 1) < 0.3
    # estimates lie on the grid 2 n / reps - 1
    assert np.allclose((x + 1) * reps / 2, np.round((x + 1) * reps / 2))


def test_from_given_terms_matches_pipeline():
    w = wl.random_batch(611, B=2, n=4, n_gates=20, n_symbols=2, K=2)
    prog = orc.Program(w.program_blob())
    obs = orc.Observables(w.observable_blob())
    th = w.theta.astype(np.float64)
    rows = []
    for b in range(w.B):
        v = []
        for k in range(w.K):
            for c, fac in w.observables[b][k]:
                if fac:
                    v.append(orc.expectation(prog, th, orc.Observables(observable_blob([[[(1.0, fac)]]] * w.B)))[b, 0])
        rows.append(v)
    Kt = max(len(v) for v in rows)
    te = np.zeros((w.B, Kt), np.float64)
    for b, v in enumerate(rows):
        te[b, :len(v)] = v
    a = orc.sampled_expectation(prog, th, obs, 300, 9)
    # the pipeline uses fp64 term values, the other path their float32
    # rounding: a shot differs only if a draw falls between the two
    # thresholds, so the two estimates agree to within a few shots
    b_ = orc.sampled_from_terms(obs, te.astype(np.float32), 300, 9)
    assert np.abs(a - b_).max() <= 4 * 2.0 / 300 * max(abs(c) for r in w.observables for t in r for c, _ in t)
