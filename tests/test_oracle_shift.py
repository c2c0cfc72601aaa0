"""Pins of the oracle's parameter-shift and finite-difference gradients
(Sec. "Parameter shift methods", eq. parshift_grad; Sec. "Finite difference
methods", eq. central_diff; shared symbols by the chain rule, eq.
chain_rule).  The shift rule is checked against the adjoint method (an
independent algorithm), against closed forms of one-gate circuits for every
kind of generator, and, with sampled expectations, against the sampled
expectation of the shifted circuits built here by hand; central differences
against their closed form on RX and against the adjoint within O(eps^2)."""
import math

import numpy as np
import pytest

from oracle import oracle as orc
from paper_2003_02989_amd import workloads as wl
from paper_2003_02989_amd.circuits import Circuit, const, observable_blob, program_blob, sym

# every opcode with a two-term rule (fSim only with a constant theta)
OPS = [o for o in wl.ONE_Q + wl.TWO_Q if o != "FSIM"]


def _random_supported(rng, n, n_gates, S):
    c = wl.random_circuit(rng, n, n_gates, S, p_symbolic=0.8, ops=OPS)
    # fSim with a symbolic phi and Pauli exponentials of weight 0..3
    c.add("FSIM", (0, n - 1), [const(float(rng.uniform(-3, 3))), sym(int(rng.integers(0, S)), 1.3, 0.2)])
    for w in range(4):
        qs = rng.choice(n, size=min(w, n), replace=False)
        fac = [(int(q), "XYZ"[int(rng.integers(0, 3))]) for q in qs]
        c.add_pauli_exp(fac, sym(int(rng.integers(0, S)), float(rng.uniform(-2, 2)), float(rng.uniform(-1, 1))))
    return c


@pytest.mark.parametrize("seed", range(3))
def test_shift_rule_equals_adjoint(seed):
    rng = np.random.default_rng(700 + seed)
    S, K = 4, 2
    circuits = [_random_supported(rng, n, 16, S) for n in (3, 4, 5)]
    obs = [wl.random_observables(rng, c.n, K) for c in circuits]
    prog = orc.Program(program_blob(circuits, S))
    o = orc.Observables(observable_blob(obs))
    theta = rng.uniform(-3, 3, size=(3, S))
    up = rng.standard_normal((3, K))
    g_ps = orc.param_shift_grad(prog, theta, o, up)
    g_adj = orc.adjoint_grad(prog, theta, o, up)
    assert np.abs(g_ps - g_adj).max() < 1e-10


@pytest.mark.parametrize("name,f", [
    # <Z> after one gate on |0> (or |+> |+> for fSim) as a function of eta
    ("RX", lambda e: math.cos(e)),
    ("XPOW", lambda t: math.cos(math.pi * t)),
    ("YPOW", lambda t: math.cos(math.pi * t)),
    ("PAULIEXP_X", lambda e: math.cos(2 * e)),
    ("PAULIEXP_Y", lambda e: math.cos(2 * e)),
    ("FSIM_PHI", lambda p: (1 + math.cos(p)) / 2),   # <XX> of (1, 1, 1, e^{-i phi}) / 2
])
def test_shift_rule_closed_forms(name, f):
    scale, offset, th = -1.7, 0.4, 0.9
    c = Circuit(2 if name == "FSIM_PHI" else 1)
    p = sym(0, scale, offset)
    if name == "FSIM_PHI":
        c.add("H", 0).add("H", 1).add("FSIM", (0, 1), [const(0.0), p])
        ob = [(1.0, [(0, "X"), (1, "X")])]
    elif name.startswith("PAULIEXP"):
        c.add_pauli_exp([(0, name[-1])], p)
        ob = [(1.0, [(0, "Z")])]
    else:
        c.add(name, 0, [p])
        ob = [(1.0, [(0, "Z")])]
    prog = orc.Program(program_blob([c], 1))
    o = orc.Observables(observable_blob([[ob]]))
    g = orc.param_shift_grad(prog, np.array([[th]]), o, np.ones((1, 1)))[0, 0]
    eta, h = scale * th + offset, 1e-5
    want = scale * (f(eta + h) - f(eta - h)) / (2 * h)
    assert abs(g - want) < 1e-8, (g, want)


def test_shared_symbol_adds_over_occurrences():
    # RX(theta) RX(theta) |0> = RX(2 theta) |0>: d<Z>/d theta = -2 sin(2 theta)
    c = Circuit(1).add("RX", 0, [sym(0)]).add("RX", 0, [sym(0)])
    th = 0.37
    g = orc.param_shift_grad(orc.Program(program_blob([c], 1)), np.array([[th]]),
                             orc.Observables(observable_blob([[[(1.0, [(0, "Z")])]]])), np.ones((1, 1)))
    assert abs(g[0, 0] + 2 * math.sin(2 * th)) < 1e-13


def test_fsim_theta_has_no_two_term_rule():
    c = Circuit(2).add("FSIM", (0, 1), [sym(0), const(0.3)])
    with pytest.raises(orc.OracleError):
        orc.param_shift_grad(orc.Program(program_blob([c], 1)), np.zeros((1, 1)),
                             orc.Observables(observable_blob([[[(1.0, [(0, "Z")])]]])), np.ones((1, 1)))


def _shifted_batch(circuits, deltas_of):
    """The shifted circuits of every row in the order (row, occurrence in gate
    and parameter order, + then -), built here by moving one parameter's
    offset, with the shift rule's (delta, factor) from deltas_of(name, j)."""
    rows, meta = [], []
    for b, c in enumerate(circuits):
        for i, (name, qubits, params, matrix) in enumerate(c.gates):
            for j, (s, scale, offset) in enumerate(params):
                if s < 0:
                    continue
                delta, factor = deltas_of(name, j)
                for sign in (1, -1):
                    nc = Circuit(c.n)
                    nc.gates = list(c.gates)
                    ps = list(params)
                    ps[j] = (s, scale, offset + sign * delta)
                    nc.gates[i] = (name, qubits, tuple(ps), matrix)
                    rows.append(nc)
                    meta.append((b, s, sign * scale * factor))
    return rows, meta


def _rule(name, j):
    if name in ("RX", "RY", "RZ", "RZZ"):
        return math.pi / 2, 0.5
    if name == "PAULIEXP":
        return math.pi / 4, 1.0
    if name == "FSIM":
        return math.pi / 2, 0.5
    return 0.5, math.pi / 2


@pytest.mark.parametrize("reps", [0, 40])
def test_shift_rule_from_shifted_circuits(reps):
    # the sampled shift rule uses, for shifted circuit e, the sampled
    # expectation of row e of the batch of shifted circuits
    rng = np.random.default_rng(711)
    S, K = 3, 2
    circuits = [_random_supported(rng, n, 8, S) for n in (3, 2)]
    obs = [wl.random_observables(rng, c.n, K) for c in circuits]
    theta = rng.uniform(-3, 3, size=(2, S))
    up = rng.standard_normal((2, K))
    g = orc.param_shift_grad(orc.Program(program_blob(circuits, S)), theta,
                             orc.Observables(observable_blob(obs)), up, reps=reps, seed=77)
    rows, meta = _shifted_batch(circuits, _rule)
    sp = orc.Program(program_blob(rows, S))
    th_rows = np.array([theta[b] for b, _, _ in meta])
    so = orc.Observables(observable_blob([obs[b] for b, _, _ in meta]))
    f = orc.expectation(sp, th_rows, so) if reps == 0 else orc.sampled_expectation(sp, th_rows, so, reps, 77)
    want = np.zeros_like(g)
    for e, (b, s, w) in enumerate(meta):
        want[b, s] += w * (f[e] @ up[b])
    assert np.abs(g - want).max() < 1e-11


def test_sampled_shift_rule_is_unbiased():
    # mean over seeds of the sampled shift-rule gradient -> the exact one,
    # within 5 standard errors of the spread across seeds
    rng = np.random.default_rng(712)
    S = 2
    c = _random_supported(rng, 3, 6, S)
    obs = [wl.random_observables(rng, 3, 1)]
    prog = orc.Program(program_blob([c], S))
    o = orc.Observables(observable_blob(obs))
    theta = rng.uniform(-3, 3, size=(1, S))
    up = np.ones((1, 1))
    exact = orc.param_shift_grad(prog, theta, o, up)
    runs = np.array([orc.param_shift_grad(prog, theta, o, up, reps=200, seed=s)[0] for s in range(60)])
    se = runs.std(axis=0, ddof=1) / math.sqrt(len(runs))
    assert np.all(np.abs(runs.mean(axis=0) - exact[0]) <= 5 * se + 1e-12)
    assert np.all(runs.std(axis=0) > 0)


def test_central_difference_closed_form():
    # <Z> of RX(s theta + o)|0> is cos(s theta + o); its central difference
    # of step eps is -sin(s theta + o) sin(s eps) / eps exactly
    s, off, th, eps = 1.3, -0.2, 0.8, 1e-2
    c = Circuit(1).add("RX", 0, [sym(0, s, off)])
    g = orc.finite_diff_grad(orc.Program(program_blob([c], 2)), np.array([[th, 0.5]]),
                             orc.Observables(observable_blob([[[(1.0, [(0, "Z")])]]])), np.ones((1, 1)), eps)
    assert abs(g[0, 0] + math.sin(s * th + off) * math.sin(s * eps) / eps) < 1e-12
    assert g[0, 1] == 0.0  # a symbol no gate uses


def test_central_difference_converges_to_adjoint():
    rng = np.random.default_rng(713)
    S, K = 3, 2
    circuits = [wl.random_circuit(rng, 4, 16, S, p_symbolic=0.8) for _ in range(2)]
    obs = [wl.random_observables(rng, 4, K) for _ in range(2)]
    prog = orc.Program(program_blob(circuits, S))
    o = orc.Observables(observable_blob(obs))
    theta = rng.uniform(-3, 3, size=(2, S))
    up = rng.standard_normal((2, K))
    exact = orc.adjoint_grad(prog, theta, o, up)
    e1 = np.abs(orc.finite_diff_grad(prog, theta, o, up, 1e-2) - exact).max()
    e2 = np.abs(orc.finite_diff_grad(prog, theta, o, up, 5e-3) - exact).max()
    assert e1 < 5e-2 and e2 < e1
    # truncation error O(eps^2): halving eps divides it by ~4
    assert 3.0 < e1 / e2 < 5.0


def test_noisy_rows_shift_rule_equals_adjoint():
    # shifted circuits of a trajectory keep its channel draws
    w = wl.with_noise(wl.random_batch(714, B=2, n=3, n_gates=8, n_symbols=2, K=1, ops=["RX", "RY", "CNOT", "RZZ"]),
                      0.2, 3)
    orc.set_noise_seed(5)
    try:
        prog = orc.Program(w.program_blob())
        o = orc.Observables(w.observable_blob())
        th = w.theta.astype(np.float64)
        up = w.upstream.astype(np.float64)
        assert np.abs(orc.param_shift_grad(prog, th, o, up) - orc.adjoint_grad(prog, th, o, up)).max() < 1e-10
    finally:
        orc.set_noise_seed(0)
