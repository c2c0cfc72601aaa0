"""The device matrix builder against the host gate table: every matrix block
the builder writes (fused products, W^dagger and dW/deta of the reverse
sweep, their storage as diagonals, (a, b) pairs or excitation-preserving
entries, and the row phase folded into the first qubit's product-init
matrix) equals the product formed on the host from tq_gate_matrix, whose
matrices and derivatives tests/test_gate_table_cpu.py pins to the oracle."""
import numpy as np
import pytest
import torch

from gpu_util import dev, say
from paper_2003_02989_amd import tq
from paper_2003_02989_amd import workloads as wl
from paper_2003_02989_amd.circuits import OPS, Circuit, sym

pytestmark = pytest.mark.gpu
SWAP_Q = [0, 2, 1, 3]  # |ab> -> |ba> on the local index 2a + b


def eta_of(gate, theta_row):
    _, _, params, _ = gate
    return [sc * float(theta_row[s]) + off if s >= 0 else off for s, sc, off in params]


def expected_block(grp, circuit, theta_row, nent):
    out = np.full(nent, np.nan, complex)
    gates = circuit.gates
    phase = 0.0
    for gate in gates:
        phase += tq.gate_matrix(OPS[gate[0]][0], eta_of(gate, theta_row), explicit=gate[3])[1]
    for kind, dim, storage, which, off, members in grp["tasks"]:
        acc = np.eye(dim, dtype=complex)
        for gi, swapped, form in members:
            gate = gates[gi]
            code = OPS[gate[0]][0]
            m, _ = tq.gate_matrix(code, eta_of(gate, theta_row), explicit=gate[3], cblock=bool(form),
                                  deriv=kind == 2, which=which)
            if m.shape[0] != dim:
                continue
            if dim == 4 and swapped:
                m = m[np.ix_(SWAP_Q, SWAP_Q)]
            if kind == 1:
                acc = m.conj().T
            elif kind == 2 or len(members) == 1:
                acc = m
            else:
                acc = m @ acc
        if storage == 0:
            v = acc.ravel()
        elif storage == 1:
            v = np.diag(acc).copy()
        elif storage in (2, 3):
            v = np.array([acc[0, 0], (-1.0 if storage == 3 else 1.0) * acc[0, dim - 1]])
        else:
            v = acc.ravel()[[0, 5, 6, 9, 10, 15]]
        if grp["n"] > 0 and off == grp["init_mat"][0]:
            v = v * np.exp(1j * phase)
        out[off:off + len(v)] = v
    return out


def check(w, **opts):
    p = tq.Program(w.program_blob(), **opts)
    plan = tq.describe(p)
    th = dev(w.theta) if w.n_symbols else None
    got = tq.build_matrices(p, th).cpu().numpy()
    torch.cuda.synchronize()
    o = 0
    worst = 0.0
    for grp in plan["groups"]:
        nb = max(grp["mat_block"], 1)
        for r, b in enumerate(grp["row_ids"]):
            blk = got[o + r * nb: o + (r + 1) * nb]
            ref = expected_block(grp, w.circuits[b], w.theta[b] if w.n_symbols else [], nb)
            known = ~np.isnan(ref)
            err = np.abs(blk[known] - ref[known])
            if err.size:
                worst = max(worst, float(err.max()))
            bad = np.nonzero(err > 1e-12)[0]
            assert bad.size == 0, (w.name, b, np.nonzero(known)[0][bad][:8], blk[known][bad][:4], ref[known][bad][:4])
        o += len(grp["row_ids"]) * nb
    return worst


@pytest.mark.parametrize("seed", range(3))
def test_builder_random_circuits(seed):
    # every opcode, fused products, reverse daggers and derivatives
    w = wl.random_batch(4100 + seed, B=4, n=6, n_gates=60, n_symbols=4, K=1, hetero=True)
    say("builder random", seed, "max error", check(w))


def test_builder_yy_power():
    c = Circuit(2).add("H", 0).add("RY", 1, [0.4]).add("YYPOW", (0, 1), [sym(0)]).add("XXPOW", (1, 0), [sym(0, -0.7, 0.2)])
    w = wl.Workload("yy", [c], 1, np.array([[0.37]], np.float32), [[[(1.0, [(0, "Z")])]]], np.ones((1, 1), np.float32))
    say("builder YY max error", check(w))
