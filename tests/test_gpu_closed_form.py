"""Expectations of product states at full size (up to 30 qubits) against a
closed form that does not go through the oracle.  RY(t) then RZ(f) on |0>
leaves a qubit with Bloch vector (sin t cos f, sin t sin f, cos t); on a
product state a Pauli string's expectation is its coefficient times the
product of its factors' Bloch components.

Error bound: the state is stored in complex64 (a relative rounding of about
6e-8 per stored value, a few roundings deep after one fused pass), and every
term's expectation is formed in fp64 from the stored amplitudes, so a term
deviates by at most a few 1e-7 of its |coefficient|; the fp32 output adds a
relative 6e-8.  The tolerance is 1e-6 sum |c| + 1e-6 per observable."""
import numpy as np
import pytest
import torch

from gpu_util import dev, say
from paper_2003_02989_amd import tq
from paper_2003_02989_amd.circuits import Circuit, observable_blob, program_blob, sym
from paper_2003_02989_amd.workloads import random_pauli_strings

pytestmark = pytest.mark.gpu


def bloch(t, f):
    return {"X": np.sin(t) * np.cos(f), "Y": np.sin(t) * np.sin(f), "Z": np.cos(t)}


def closed_form(terms, th, ph):
    b = [bloch(th[q], ph[q]) for q in range(len(th))]
    return sum(c * np.prod([b[q][p] for q, p in factors]) for c, factors in terms)


def observable_set(kind, n, rng):
    if kind == "c5_shape":  # one observable of 200 random X/Y/Z strings
        return [random_pauli_strings(rng, n, 200)]
    if kind == "sixteen":  # sixteen observables, 650 strings over all
        return [random_pauli_strings(rng, n, 200)] + [random_pauli_strings(rng, n, 30) for _ in range(15)]
    # Z-only: a QAOA-shaped cut observable (30 Z_i Z_j and a constant)
    pairs = [rng.choice(n, size=2, replace=False) for _ in range(30)]
    return [[(-0.5, [(int(a), "Z"), (int(b), "Z")]) for a, b in pairs] + [(15.0, [])]]


@pytest.mark.parametrize("kind", ["c5_shape", "sixteen", "zz"])
@pytest.mark.parametrize("specialize", [False, True])
@pytest.mark.parametrize("n,B", [(20, 64), (30, 1)])
def test_product_state_expectations(n, B, specialize, kind):
    rng = np.random.default_rng(900 + n)
    obs = observable_set(kind, n, rng)
    c = Circuit(n)
    for q in range(n):
        c.add("RY", q, [sym(q)])
        c.add("RZ", q, [sym(n + q)])
    theta = rng.uniform(0.0, 2 * np.pi, size=(B, 2 * n)).astype(np.float32)
    say("product state n", n, "B", B, "observables", kind, "specialize", specialize)
    p = tq.Program(program_blob([c] * B, 2 * n), specialize=specialize)
    o = tq.Observables(observable_blob([obs] * B))
    e = tq.expectation(p, dev(theta, torch.float32), o).cpu().numpy()
    ob = tq.describe(p)["groups"][0]["obs"]
    # the route taken: the Z-only stream, else (specialize = 1) the
    # expectation passes generated for the terms, else the table-driven kernel
    if kind == "zz":
        assert ob["diag"] == 1
    else:
        assert bool(ob["exp_passes"]) == specialize
    th = theta.astype(np.float64)
    ref = np.array([[closed_form(terms, th[b, :n], th[b, n:]) for terms in obs] for b in range(B)])
    tol = 1e-6 * np.array([sum(abs(cf) for cf, _ in terms) for terms in obs]) + 1e-6
    err = np.abs(e - ref)
    say("max |error|", float(err.max()), "max error / tolerance", float((err / tol).max()))
    assert np.all(err <= tol)
