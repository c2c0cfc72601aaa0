"""Pins of the oracle's gate table: unitarity, agreement with gates built
independently from their generators by matrix exponentials, the algebraic
identities of the opcode set, and derivatives against finite differences."""
import math

import numpy as np
import pytest

from oracle import dense
from oracle import oracle as orc
from paper_2003_02989_amd.circuits import OPS

rng = np.random.default_rng(7)


def _params(name):
    return [float(x) for x in rng.uniform(-3, 3, size=OPS[name][2])]


@pytest.mark.parametrize("name", [n for n in OPS if not n.startswith("MATRIX") and OPS[n][1] is not None and n != "PCHAN"])
def test_gate_matches_generator_definition(name):
    for _ in range(5):
        p = _params(name)
        m = orc.gate_matrix(OPS[name][0], p)
        ref = dense.gate(name, p)
        assert np.abs(m - ref).max() < 1e-13, name
        d = m.shape[0]
        assert np.abs(m.conj().T @ m - np.eye(d)).max() < 1e-14


def test_explicit_matrices_pass_through():
    for op, d in ((OPS["MATRIX1"][0], 2), (OPS["MATRIX2"][0], 4)):
        u = np.linalg.qr(rng.standard_normal((d, d)) + 1j * rng.standard_normal((d, d)))[0]
        assert np.abs(orc.gate_matrix(op, [], u) - u).max() == 0


def G(name, *p):
    return orc.gate_matrix(OPS[name][0], list(p))


def test_identities():
    X, Y, Z = dense.PX, dense.PY, dense.PZ
    assert np.allclose(G("RX", math.pi), -1j * X, atol=1e-15)
    assert np.allclose(G("XPOW", 1.0), X, atol=1e-15)
    assert np.allclose(G("YPOW", 1.0), Y, atol=1e-15)
    assert np.allclose(G("ZPOW", 1.0), Z, atol=1e-15)
    assert np.allclose(G("ZZPOW", 1.0), np.kron(Z, Z), atol=1e-15)
    assert np.allclose(G("XXPOW", 1.0), np.kron(X, X), atol=1e-15)
    assert np.allclose(G("CZPOW", 1.0), G("CZ"), atol=1e-15)
    assert np.allclose(G("CNOTPOW", 1.0), G("CNOT"), atol=1e-15)
    sx, sy, sw = G("SQRTX"), G("SQRTY"), G("SQRTW")
    W = (X + Y) / math.sqrt(2)
    assert np.allclose(sx @ sx, X, atol=1e-15)
    assert np.allclose(sy @ sy, Y, atol=1e-15)
    assert np.allclose(sw @ sw, W, atol=1e-15)
    # sqrt(W) = Z^(1/4) sqrt(X) Z^(-1/4)
    assert np.allclose(sw, G("ZPOW", 0.25) @ sx @ G("ZPOW", -0.25), atol=1e-15)
    # printed entries of the three random-circuit gates
    h = 0.5
    assert np.allclose(sx, [[h + h * 1j, h - h * 1j], [h - h * 1j, h + h * 1j]], atol=1e-15)
    assert np.allclose(sy, [[h + h * 1j, -h - h * 1j], [h + h * 1j, h + h * 1j]], atol=1e-15)
    r = 1 / math.sqrt(2)
    assert np.allclose(sw, [[h + h * 1j, -1j * r], [r, h + h * 1j]], atol=1e-15)
    assert np.allclose(G("FSIM", 0.0, 0.0), np.eye(4), atol=1e-15)
    f = G("FSIM", math.pi / 2, math.pi / 6)
    assert np.allclose(f[1:3, 1:3], [[0, -1j], [-1j, 0]], atol=1e-15)
    assert np.isclose(f[3, 3], np.exp(-1j * math.pi / 6))
    # RZ is diag(e^{-i t/2}, e^{i t/2}); ZPOW is diag(1, e^{i pi t})
    t = 0.7
    assert np.allclose(G("RZ", t), np.diag([np.exp(-0.5j * t), np.exp(0.5j * t)]), atol=1e-15)
    assert np.allclose(G("ZPOW", t), np.diag([1, np.exp(1j * math.pi * t)]), atol=1e-15)
    assert np.allclose(G("RZZ", t), np.diag(np.exp(-0.5j * t * np.array([1, -1, -1, 1]))), atol=1e-15)
    # CNOT flips the second qubit when the first is 1 (local index 2*a + b)
    assert np.allclose(G("CNOT"), [[1, 0, 0, 0], [0, 1, 0, 0], [0, 0, 0, 1], [0, 0, 1, 0]])
    assert np.allclose(G("SWAP"), [[1, 0, 0, 0], [0, 0, 1, 0], [0, 1, 0, 0], [0, 0, 0, 1]])


def test_periodicity():
    for t in (0.3, -1.1):
        assert np.allclose(G("RX", t + 4 * math.pi), G("RX", t), atol=1e-13)
        assert np.allclose(G("RX", t + 2 * math.pi), -G("RX", t), atol=1e-13)
        for name in ("XPOW", "YPOW", "ZPOW", "CZPOW", "CNOTPOW", "XXPOW", "YYPOW", "ZZPOW"):
            assert np.allclose(G(name, t + 2), G(name, t), atol=1e-13), name


@pytest.mark.parametrize("name", [n for n, v in OPS.items() if v[2] > 0 and v[1] is not None and n != "PCHAN"])
def test_derivative_matches_central_difference(name):
    op, _, npar = OPS[name]
    h = 1e-6
    for which in range(npar):
        p = _params(name)
        dm = orc.gate_dmatrix(op, p, which)
        pp, pm = list(p), list(p)
        pp[which] += h
        pm[which] -= h
        fd = (orc.gate_matrix(op, pp) - orc.gate_matrix(op, pm)) / (2 * h)
        assert np.abs(dm - fd).max() < 1e-8, (name, which)


def test_splitmix64_published_vector():
    # first outputs of SplitMix64 started from state 0 (reference
    # implementation of Steele, Lea and Flood, as distributed with xoshiro)
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]
    assert [orc.splitmix64(0, i) for i in range(4)] == want
