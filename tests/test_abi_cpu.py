"""Host-side checks of the C ABI, no GPU needed: libtq.so loads, exports
every function include/tq.h declares, and rejects malformed input on the
host before any device call."""
import ctypes
import os
import re
import struct

import pytest

from paper_2003_02989_amd import tq
from paper_2003_02989_amd import workloads as wl
from paper_2003_02989_amd.circuits import Circuit, observable_blob, program_blob, sym

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "tq.h")).read()
    return sorted(set(re.findall(r"\b(tq_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 14
    L = tq.lib()
    for n in names:
        assert hasattr(L, n), n


def create(blob, **kw):
    return tq.Program(blob, **kw)


def status_of(fn):
    with pytest.raises(tq.TQError) as e:
        fn()
    return e.value.status


def test_program_info_roundtrip():
    w = wl.random_batch(3, B=5, n=6, n_gates=12, n_symbols=3, hetero=True)
    p = create(w.program_blob())
    assert (p.B, p.S, p.max_qubits) == (5, 3, max(c.n for c in w.circuits))
    assert p.qubits == [c.n for c in w.circuits]


def gate_blob(op, nq, npar, qubits, params=(), n=3, S=1):
    body = struct.pack("<HBB", op, nq, npar) + struct.pack(f"<{len(qubits)}I", *qubits)
    for s, scale, off in params:
        body += struct.pack("<idd", s, scale, off)
    return b"TQP1" + struct.pack("<III", 1, 1, S) + struct.pack("<II", n, 1) + body


def test_bad_programs_are_rejected_on_the_host():
    good = gate_blob(5, 1, 1, [0], [(0, 1.0, 0.0)])
    create(good)
    assert status_of(lambda: create(b"XXXX" + good[4:])) == tq.TQ_E_INVALID
    assert status_of(lambda: create(good[:-3])) == tq.TQ_E_INVALID
    assert status_of(lambda: create(good + b"\0")) == tq.TQ_E_INVALID
    assert status_of(lambda: create(gate_blob(5, 1, 1, [3], [(0, 1.0, 0.0)]))) == tq.TQ_E_INVALID  # qubit >= n
    assert status_of(lambda: create(gate_blob(11, 2, 0, [1, 1]))) == tq.TQ_E_INVALID  # repeated qubit
    assert status_of(lambda: create(gate_blob(5, 1, 1, [0], [(1, 1.0, 0.0)]))) == tq.TQ_E_INVALID  # symbol >= S
    assert status_of(lambda: create(gate_blob(5, 2, 1, [0, 1], [(0, 1.0, 0.0)]))) == tq.TQ_E_INVALID  # arity
    assert status_of(lambda: create(gate_blob(99, 1, 0, [0]))) == tq.TQ_E_UNSUPPORTED  # opcode
    big = b"TQP1" + struct.pack("<III", 1, 1, 0) + struct.pack("<II", 33, 0)
    assert status_of(lambda: create(big)) == tq.TQ_E_UNSUPPORTED
    assert status_of(lambda: create(good, max_tile_qubits=20)) == tq.TQ_E_INVALID


def test_bad_observables_are_rejected():
    ok = observable_blob([[[(1.0, [(0, "Z")])]]])
    tq.Observables(ok)
    bad_code = ok[:-1] + b"\x07"
    assert status_of(lambda: tq.Observables(bad_code)) == tq.TQ_E_INVALID
    dup = observable_blob([[[(1.0, [(0, "Z"), (0, "X")])]]])
    assert status_of(lambda: tq.Observables(dup)) == tq.TQ_E_INVALID
    assert status_of(lambda: tq.Observables(ok[:-2])) == tq.TQ_E_INVALID


def test_compute_calls_validate_before_touching_the_device():
    L = tq.lib()
    c = Circuit(2).add("RX", 0, [sym(0)]).add("CNOT", (0, 1))
    p = create(program_blob([c, c], 1))
    o = tq.Observables(observable_blob([[[(1.0, [(1, "Z")])]]] * 2))
    o1 = tq.Observables(observable_blob([[[(1.0, [(1, "Z")])]]]))
    o3 = tq.Observables(observable_blob([[[(1.0, [(2, "Z")])]]] * 2))
    fake = ctypes.c_void_p(16)
    assert L.tq_expectation(p._h, fake, o._h, None, None) == tq.TQ_E_INVALID  # out NULL
    assert L.tq_expectation(p._h, None, o._h, fake, None) == tq.TQ_E_INVALID  # theta NULL with S > 0
    assert L.tq_expectation(p._h, fake, o1._h, fake, None) == tq.TQ_E_INVALID  # batch mismatch
    assert L.tq_expectation(p._h, fake, o3._h, fake, None) == tq.TQ_E_INVALID  # qubit >= n_b
    assert b"qubit" in L.tq_last_error()
    assert L.tq_sample(p._h, fake, -1, 0, fake, None) == tq.TQ_E_INVALID
    assert L.tq_amplitudes(p._h, fake, None, 3, fake, None) == tq.TQ_E_INVALID
    assert L.tq_adjoint_grad(p._h, fake, o._h, None, fake, None, None) == tq.TQ_E_INVALID
    assert L.tq_simulate_state(p._h, fake, None, None) == tq.TQ_E_INVALID
    assert L.tq_sample_from_state(fake, 1, 40, 1, 0, fake, None) == tq.TQ_E_INVALID
    assert L.tq_program_create(b"", 0, None, None) == tq.TQ_E_INVALID
    # empty work is a no-op that needs no device
    assert L.tq_sample(p._h, fake, 0, 0, None, None) == tq.TQ_OK
    assert L.tq_sample_from_state(None, 0, 3, 5, 0, None, None) == tq.TQ_OK


def test_version():
    assert tq.lib().tq_version().startswith(b"tq ")


def test_specialized_kernels_compile_for_gfx950():
    # the kernels generated per circuit structure compile with hipRTC for
    # gfx950 (no device needed): the two resident configurations, random
    # resident structures over the whole opcode set, and the forward and
    # reverse tile passes of a 14-qubit random structure
    # (and the QAOA and VQE structures: phase classes, diagonal runs)
    for w in (wl.c1_hea(), wl.c2_qnn(B=4),
              wl.random_batch(6601, B=3, n=10, n_gates=60, n_symbols=5, K=3, hetero=True),
              wl.random_batch(1412, B=2, n=14, n_gates=60, n_symbols=5, K=2),
              wl.c3_qaoa(B=2), wl.c5_vqe(B=2, layers=3)):
        p = create(w.program_blob(), specialize=True)
        tq.specialize(p, "gfx950")
    # a program without the option has nothing to compile
    tq.specialize(create(wl.c2_qnn(B=2).program_blob()), "gfx950")


def test_specialize_option_is_validated():
    blob = wl.c1_hea().program_blob()
    opt = tq._Options(0, 0, 1, 0, 2)
    h = ctypes.c_void_p()
    assert tq.lib().tq_program_create(blob, len(blob), ctypes.byref(opt), ctypes.byref(h)) == tq.TQ_E_INVALID


def test_pauli_exponential_is_lowered_and_validated():
    # exp(-i eta P) becomes gates of the fixed table: X -> H, Y -> RX(pi/2) on
    # both sides, weight 3 -> one CNOT each side of RZZ; weight 1 -> RX, RY or
    # RZ; weight 0 -> RZ and ZPOW on qubit 0
    c = Circuit(4).add_pauli_exp([(0, "X"), (2, "Y"), (3, "Z")], sym(0, 0.5))
    d = tq.describe(create(program_blob([c], 1)))
    assert d["groups"][0]["gates"] == 2 + 1 + 1 + 1 + 2
    for fac, ng in (([(1, "Z")], 1), ([(1, "X")], 1), ([(2, "Y")], 1), ([], 2), ([(0, "Z"), (3, "Z")], 1),
                    ([(0, "X"), (3, "Y")], 5),
                    ([(q, "Z") for q in range(4)], 5)):
        d = tq.describe(create(program_blob([Circuit(4).add_pauli_exp(fac, sym(0))], 1)))
        assert d["groups"][0]["gates"] == ng, fac
    # same structure for rows that differ only in the exponential's scale
    rows = [Circuit(3).add_pauli_exp([(0, "X"), (1, "Z")], sym(0, s)) for s in (0.3, -1.0)]
    assert len(tq.describe(create(program_blob(rows, 1)))["groups"]) == 1

    def blob(qubits, codes, np_=1, n=4):
        return (b"TQP1" + struct.pack("<III", 1, 1, 1) + struct.pack("<II", n, 1)
                + struct.pack("<HBB", 26, len(qubits), np_) + struct.pack(f"<{len(qubits)}I", *qubits)
                + b"".join(struct.pack("<idd", 0, 1.0, 0.0) for _ in range(np_)) + bytes(codes))
    create(blob([0, 1], [1, 3]))
    assert status_of(lambda: create(blob([0, 0], [1, 3]))) == tq.TQ_E_INVALID  # repeated qubit
    assert status_of(lambda: create(blob([0, 4], [1, 3]))) == tq.TQ_E_INVALID  # qubit >= n
    assert status_of(lambda: create(blob([0, 1], [1, 4]))) == tq.TQ_E_INVALID  # Pauli code
    assert status_of(lambda: create(blob([0, 1], [1, 3], np_=2))) == tq.TQ_E_INVALID  # parameters
    assert status_of(lambda: create(blob([0, 1], [1, 3])[:-1])) == tq.TQ_E_INVALID  # truncated
    assert status_of(lambda: create(blob([0, 1, 2, 3, 0], [1, 1, 1, 1, 1]))) == tq.TQ_E_INVALID  # longer than n


def test_channels_validated_and_seed_entry_points():
    from paper_2003_02989_amd.circuits import const
    create(program_blob([Circuit(2).add("PCHAN", 1, [0.1, 0.2, 0.3])], 0))
    for params in ([0.5, 0.6, 0.0], [-0.1, 0.0, 0.0]):
        assert status_of(lambda: create(program_blob([Circuit(2).add("PCHAN", 0, params)], 0))) == tq.TQ_E_INVALID
    assert status_of(lambda: create(program_blob([Circuit(2).add("PCHAN", 0, [sym(0), 0.0, 0.0])], 1))) \
        == tq.TQ_E_INVALID
    L = tq.lib()
    assert L.tq_program_set_noise_seed(None, 1) == tq.TQ_E_INVALID
    p = create(program_blob([Circuit(2).add("PCHAN", 1, [0.1, 0.2, 0.3])], 0))
    assert L.tq_program_set_noise_seed(p._h, 77) == tq.TQ_OK
    fake = ctypes.c_void_p(16)
    assert L.tq_row_mean(fake, 2, 0, 1, fake, None) == tq.TQ_E_INVALID  # R < 1
    assert L.tq_row_mean(None, 2, 3, 1, fake, None) == tq.TQ_E_INVALID  # in NULL
    assert L.tq_row_mean(None, 0, 3, 1, None, None) == tq.TQ_OK  # no work
    # a noisy structure's generated kernels compile for gfx950
    w = wl.with_noise(wl.random_batch(1413, B=2, n=14, n_gates=30, n_symbols=3, K=1), 0.05, 2)
    tq.specialize(create(w.program_blob(), specialize=True), "gfx950")


def test_shift_rule_occurrences_and_validation():
    # every symbolic blob parameter is one occurrence; the global phase of a
    # weight-0 Pauli exponential drives two lowered slots as one occurrence,
    # and the same lowered gates written out by hand stay two occurrences
    # (a structure of its own)
    from paper_2003_02989_amd.circuits import const
    c1 = Circuit(2).add("RX", 0, [sym(0)]).add_pauli_exp([], sym(1, 0.5)).add("FSIM", (0, 1), [const(0.2), sym(0)])
    c2 = Circuit(2).add("RX", 0, [sym(0)]).add("RZ", 0, [sym(1, 1.0)]).add("ZPOW", 0, [sym(1, -2 / 3.141592653589793)])
    c2.add("FSIM", (0, 1), [const(0.2), sym(0)])
    p = create(program_blob([c1, c2], 2))
    d = tq.describe(p)
    assert len(d["groups"]) == 2
    occ = [[o[:3] + [o[3], o[4]] for o in g["occurrences"]] for g in d["groups"]]
    assert [len(o) for o in occ] == [3, 4]
    g0 = occ[0]
    assert g0[0][1] == -1 and g0[0][2] == 0 and g0[0][3] == 5            # RX
    assert g0[1][1] >= 0 and g0[1][2] == 1 and g0[1][3] == 26           # exp(-i eta I): two slots
    assert g0[2][2] == 0 and g0[2][3] == 22 and g0[2][4] == 1            # fSim phi
    L = tq.lib()
    o = tq.Observables(observable_blob([[[(1.0, [(0, "Z")]), (0.5, [])]]] * 2))
    assert tq.observables_terms(o) == 1
    fake = ctypes.c_void_p(16)
    assert L.tq_sampled_expectation(p._h, fake, o._h, 0, 0, fake, None, None) == tq.TQ_E_INVALID  # reps 0
    assert L.tq_sampled_expectation(p._h, fake, o._h, 1 << 24, 0, fake, None, None) == tq.TQ_E_INVALID
    assert L.tq_sampled_expectation(p._h, fake, o._h, 10, 0, None, None, None) == tq.TQ_E_INVALID  # out NULL
    assert L.tq_param_shift_grad(p._h, fake, o._h, fake, -1, 0, fake, None) == tq.TQ_E_INVALID
    assert L.tq_param_shift_grad(p._h, fake, o._h, fake, 0, 0, None, None) == tq.TQ_E_INVALID  # grad NULL
    assert L.tq_finite_diff_grad(p._h, fake, o._h, fake, ctypes.c_double(0.0), fake, None) == tq.TQ_E_INVALID
    assert L.tq_finite_diff_grad(p._h, fake, o._h, fake, ctypes.c_double(float("nan")), fake, None) == tq.TQ_E_INVALID
    # fSim theta has no two-term rule: rejected before any device call
    c3 = Circuit(2).add("FSIM", (0, 1), [sym(0), const(0.1)])
    p3 = create(program_blob([c3], 1))
    o3 = tq.Observables(observable_blob([[[(1.0, [(0, "Z")])]]]))
    assert L.tq_param_shift_grad(p3._h, fake, o3._h, fake, 0, 0, fake, None) == tq.TQ_E_UNSUPPORTED
    assert b"shift" in L.tq_last_error()


def test_empty_batch_is_a_no_op_for_every_compute_call():
    # a program of no circuits: every compute entry point returns OK without
    # touching the device (there is none here) or its output pointers
    L = tq.lib()
    p = create(program_blob([], 2))
    o = tq.Observables(observable_blob([]))
    fake = ctypes.c_void_p(16)
    assert L.tq_simulate_state(p._h, fake, fake, None) == tq.TQ_OK
    assert L.tq_expectation(p._h, fake, o._h, fake, None) == tq.TQ_OK
    assert L.tq_adjoint_grad(p._h, fake, o._h, fake, fake, None, None) == tq.TQ_OK
    assert L.tq_sample(p._h, fake, 10, 1, fake, None) == tq.TQ_OK
    assert L.tq_amplitudes(p._h, fake, fake, 4, fake, None) == tq.TQ_OK
    assert L.tq_sampled_expectation(p._h, fake, o._h, 10, 1, fake, None, None) == tq.TQ_OK
    assert L.tq_param_shift_grad(p._h, fake, o._h, fake, 0, 0, fake, None) == tq.TQ_OK
    assert L.tq_param_shift_grad(p._h, fake, o._h, fake, 50, 3, fake, None) == tq.TQ_OK
    assert L.tq_finite_diff_grad(p._h, fake, o._h, fake, 1e-2, fake, None) == tq.TQ_OK
