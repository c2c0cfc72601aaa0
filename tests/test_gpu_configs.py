"""GPU parity on the five workload configurations: at full size where the
oracle finishes in seconds (c1, c2), on reduced sizes that still span several
tiles, and at full size on sampled rows the oracle computes one by one (c3,
c5) or against stored oracle values (c4, tests/golden/c4_n30.npz written by
tests/golden/make_c4_golden.py)."""
import os

import numpy as np
import pytest
import torch

from gpu_util import TOL_AMP, TOL_EXP, TOL_GRAD, compare, dev, gpu_outputs, oracle_outputs, say, sub_workload
from oracle import oracle as orc
from paper_2003_02989_amd import tq
from paper_2003_02989_amd import workloads as wl

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_c1_full():
    w = wl.c1_hea()
    say("c1 full")
    compare(gpu_outputs(w), oracle_outputs(w))
    w.upstream = np.random.default_rng(1).standard_normal(w.upstream.shape).astype(np.float32)
    compare(gpu_outputs(w, want=("exp", "grad")), oracle_outputs(w, want=("exp", "grad")))


def test_c2_full():
    w = wl.c2_qnn()
    say("c2 full")
    compare(gpu_outputs(w, want=("exp", "grad")), oracle_outputs(w, want=("exp", "grad")))


@pytest.mark.parametrize("name", ["c1", "c2"])
def test_specialized_resident_configs(name):
    # the structure-specialised resident kernel against the oracle, and
    # against the precompiled kernel it stands in for
    w = wl.CONFIGS[name]()
    say(name, "specialised")
    g = gpu_outputs(w, want=("exp", "grad"), specialize=True)
    compare(g, oracle_outputs(w, want=("exp", "grad")))
    base = gpu_outputs(w, want=("exp", "grad"))
    assert np.abs(g["grad"] - base["grad"]).max() <= 1e-6
    assert np.abs(g["exp"] - base["exp"]).max() <= 1e-6


def test_c3_reduced():
    w = wl.c3_qaoa(B=16, n=14)
    say("c3 reduced n=14 B=16")
    compare(gpu_outputs(w), oracle_outputs(w))


@pytest.mark.parametrize("specialize", [False, True])
def test_c3_full_sampled_rows(specialize):
    # specialize=True is the path the benchmark times: the forward passes
    # generated for the structure, the Z-only expectation stream, and with the
    # adjoint the generated H_g and reverse passes
    w = wl.c3_qaoa()
    say("c3 full n=20 B=256 specialize", specialize)
    g = gpu_outputs(w, want=("exp", "grad"), specialize=specialize)
    rows = [0, 97, 255]
    ref = oracle_outputs(sub_workload(w, rows), want=("exp", "grad"))
    gs = {"exp": g["exp"][rows], "grad": g["grad"][rows], "grad_exp": g["grad_exp"][rows]}
    say("c3 max errors: exp", float(np.abs(gs["exp"] - ref["exp"]).max()),
        "grad", float(np.abs(gs["grad"] - ref["grad"]).max()))
    compare(gs, ref)
    # invariants over every row: 0 <= <C> <= |E|
    assert np.all(g["exp"] >= -TOL_EXP) and np.all(g["exp"] <= 30 + TOL_EXP)


def test_c3_exponentials_reduced():
    # the QAOA layers built from the exponentials of the cost and mixer
    # Hamiltonians (the paper's QAOA example), every output against the oracle
    w = wl.c3_qaoa(B=16, n=14, exponentials=True)
    say("c3 by exponentials, reduced n=14 B=16")
    compare(gpu_outputs(w), oracle_outputs(w))
    compare(gpu_outputs(w, specialize=True), oracle_outputs(w))


@pytest.mark.parametrize("specialize", [False, True])
def test_c3_exponentials_full_sampled_rows(specialize):
    w = wl.c3_qaoa(exponentials=True)
    say("c3 by exponentials, full n=20 B=256 specialize", specialize)
    g = gpu_outputs(w, want=("exp", "grad"), specialize=specialize)
    rows = [0, 128, 255]
    ref = oracle_outputs(sub_workload(w, rows), want=("exp", "grad"))
    gs = {"exp": g["exp"][rows], "grad": g["grad"][rows], "grad_exp": g["grad_exp"][rows]}
    compare(gs, ref)
    # the same circuits as the RZZ / RX layers up to the parametrization:
    # exp(-i gamma (-1/2) Z Z) = RZZ(-gamma), exp(-i beta X) = RX(2 beta)
    v = wl.c3_qaoa()
    v.theta = w.theta * np.array([-1.0] * 4 + [2.0] * 4, np.float32)
    e2 = gpu_outputs(v, want=("exp",), specialize=specialize)["exp"]
    assert np.abs(e2 - g["exp"]).max() <= 2 * TOL_EXP


def test_c5_reduced():
    w = wl.c5_vqe(B=24, n=12, layers=10, n_terms=200)
    say("c5 reduced n=12 B=24")
    compare(gpu_outputs(w), oracle_outputs(w))


@pytest.mark.parametrize("specialize", [False, True])
def test_c5_full_sampled_rows(specialize):
    # specialize=True: the generated forward passes, the 200-term H_g psi in
    # several generated passes (with the expectation from the same sums) and
    # the generated reverse passes; tq_expectation alone takes the generated
    # expectation passes of the Hamiltonian
    w = wl.c5_vqe()
    say("c5 full n=16 B=4096 specialize", specialize)
    g = gpu_outputs(w, want=("exp", "grad"), specialize=specialize)
    rows = [0, 1234, 4095]
    ref = oracle_outputs(sub_workload(w, rows), want=("exp", "grad"))
    gs = {"exp": g["exp"][rows], "grad": g["grad"][rows], "grad_exp": g["grad_exp"][rows]}
    say("c5 max errors: exp", float(np.abs(gs["exp"] - ref["exp"]).max()),
        "grad", float(np.abs(gs["grad"] - ref["grad"]).max()),
        "adjoint-call exp", float(np.abs(gs["grad_exp"] - ref["exp"]).max()))
    compare(gs, ref)
    # every row: the adjoint call's expectations are the expectation call's
    assert np.abs(g["grad_exp"] - g["exp"]).max() <= 2 * TOL_EXP


def test_c5_noisy_full_sampled_rows():
    # the noisy VQE as benchmarked: depolarizing p = 0.01 after every gate,
    # 10 trajectories per circuit (40960 rows of 16 qubits), generated
    # kernels; the oracle draws the same channels for the sampled rows (rows
    # offset into the full batch)
    R = 10
    w = wl.with_noise(wl.c5_vqe(), 0.01, R)
    seed = 1000
    say("c5 noisy full n=16 rows", w.B)
    p = tq.Program(w.program_blob(), specialize=True)
    tq.set_noise_seed(p, seed)
    o = tq.Observables(w.observable_blob())
    th = dev(w.theta)
    e = tq.expectation(p, th, o).cpu().numpy()
    ge = torch.empty((w.B, w.K), dtype=torch.float32, device="cuda")
    g = tq.adjoint_grad(p, th, o, dev(w.upstream), expectations=ge).cpu().numpy()
    ge = ge.cpu().numpy()
    orc.set_noise_seed(seed)
    try:
        for r in (0, 7, 20479, 40959):
            orc.set_row_offset(r)
            ref = oracle_outputs(sub_workload(w, [r]), want=("exp", "grad"))
            say("  row", r, "exp error", float(np.abs(e[r] - ref["exp"][0]).max()),
                "grad error", float(np.abs(g[r] - ref["grad"][0]).max()))
            compare({"exp": e[[r]], "grad": g[[r]], "grad_exp": ge[[r]]}, ref)
    finally:
        orc.set_row_offset(0)
        orc.set_noise_seed(0)
    # trajectories of one circuit differ (channels applied) and their mean is
    # what tq_row_mean returns
    assert np.abs(e[0] - e[1]).max() > 0 or np.abs(e[1] - e[2]).max() > 0
    m = tq.row_mean(dev(e), R).cpu().numpy()
    assert np.abs(m - e.reshape(-1, R, w.K).astype(np.float64).mean(1)).max() < 1e-6


def _norm2_f64(st):
    # sum |psi|^2 in float64, in chunks (the n = 30 state holds 2^31 floats)
    x = st.reshape(-1).view(torch.float32)
    tot = 0.0
    for i in range(0, x.numel(), 1 << 27):
        tot += float(x[i:i + (1 << 27)].double().pow(2).sum().item())
    return tot


def _c4_check(w, amps_ref, sum_p2, norm2_ref, n, p_ref=None, **opts):
    """Amplitudes at the seeded bitstrings (relative L2 error), the state's
    norm, the sampler bit-exact on the device's own complex64 state, and the
    cross-entropy identity of the samples: with the oracle's probabilities
    p_ref when its full state is at hand, else (n = 30) with the device's
    state, which the first two checks pin to the oracle's."""
    p = tq.Program(w.program_blob(), **opts)
    bits = dev(w.extras["bitstrings"].astype(np.int64), torch.int64)
    shots = w.extras["n_shots"]
    smp, amps = tq.sample_with_amplitudes(p, None, shots, w.extras["seed"], bits)
    a = amps.cpu().numpy()[0]
    rel = np.linalg.norm(a.astype(np.complex128) - amps_ref) / np.linalg.norm(amps_ref)
    amax = np.abs(a.astype(np.complex128) - amps_ref).max() / np.abs(amps_ref).max()
    say("c4 n", n, "amplitudes: relative L2 error", rel, "max |da| / max |a|", amax)
    assert rel <= TOL_AMP
    # the one-simulation call returns what the separate calls return
    assert np.array_equal(tq.amplitudes(p, None, bits).cpu().numpy()[0], a)
    assert torch.equal(tq.sample(p, None, shots, w.extras["seed"]), smp)
    st = tq.simulate_state(p, None)
    norm2 = _norm2_f64(st)
    say("c4 n", n, "norm^2", norm2, "oracle", norm2_ref)
    assert abs(norm2 - norm2_ref) < 1e-6
    # cross-entropy identity: mean over exact samples of 2^n p(x) is 2^n sum p^2
    if p_ref is None:
        pr = (torch.abs(st[0]) ** 2).double()
        px = pr[smp[0]].cpu().numpy()
    else:
        px = p_ref[smp[0].cpu().numpy()]
    xeb = float((px * 2.0 ** n).mean())
    var = float(((px * 2.0 ** n) ** 2).mean()) - xeb ** 2
    sigma = (var / shots) ** 0.5
    say("c4 xeb", xeb, "expected", sum_p2 * 2.0 ** n, "sigma", sigma, "oracle p" if p_ref is not None else "device p")
    assert abs(xeb - sum_p2 * 2.0 ** n) < 4 * sigma
    # the sampler is bit-exact on the device's own complex64 state
    host_state = st.cpu().numpy()
    ref = orc.sample_from_state(host_state, shots, w.extras["seed"])
    assert np.array_equal(smp.cpu().numpy().astype(np.uint64), ref)
    return st


def test_c4_reduced():
    w = wl.c4_random(rows=4, cols=5, n_shots=200_000)
    say("c4 reduced n=20")
    ref = orc.simulate_state(orc.Program(w.program_blob()), np.zeros((1, 0)))[0]
    bits = w.extras["bitstrings"][0].astype(np.int64)
    p2 = np.abs(ref) ** 2
    st = _c4_check(w, ref[bits], float((p2 * p2).sum()), float(p2.sum()), 20, p_ref=p2)
    err = np.linalg.norm(st.cpu().numpy()[0].astype(np.complex128) - ref)
    say("c4 n=20 state L2 error", err)
    assert err <= TOL_AMP


def test_specialized_passes_configs():
    # tile passes compiled for the circuit structure: reduced c3 (Z-only cost
    # observable), c5 (forward and reverse passes, 60 Pauli strings) and c4
    # (fSim grid; amplitudes, norm and samples)
    w = wl.c3_qaoa(B=8, n=14)
    say("c3 reduced specialised")
    compare(gpu_outputs(w, specialize=True), oracle_outputs(w))
    w = wl.c5_vqe(B=6, n=14, layers=4, n_terms=60)
    say("c5 reduced specialised")
    compare(gpu_outputs(w, specialize=True), oracle_outputs(w))
    w = wl.c4_random(rows=3, cols=5, n_shots=100_000)
    say("c4 reduced specialised n=15")
    ref = orc.simulate_state(orc.Program(w.program_blob()), np.zeros((1, 0)))[0]
    bits = w.extras["bitstrings"][0].astype(np.int64)
    p2 = np.abs(ref) ** 2
    st = _c4_check(w, ref[bits], float((p2 * p2).sum()), float(p2.sum()), 15, p_ref=p2, specialize=True)
    assert np.linalg.norm(st.cpu().numpy()[0].astype(np.complex128) - ref) <= TOL_AMP


@pytest.mark.parametrize("specialize", [False, True])
def test_c4_full_against_golden(specialize):
    # specialize=True is the benchmark's path: 30 generated forward passes
    # over the 2^30-amplitude state (17 fixed bits per 2^13-amplitude tile)
    path = os.path.join(GOLDEN, "c4_n30.npz")
    g = np.load(path)
    w = wl.c4_random()
    assert np.array_equal(g["bitstrings"], w.extras["bitstrings"][0])
    say("c4 full n=30 specialize", specialize)
    _c4_check(w, g["amplitudes"], float(g["sum_p2"]), float(g["norm2"]), 30, specialize=specialize)


@pytest.mark.parametrize("n,n_terms", [(14, 150), (16, 200), (13, 1000)])
def test_specialized_expectation_many_terms(n, n_terms):
    # one observable of more than 64 Pauli strings, the same on every row:
    # tq_expectation runs the expectation passes generated for its terms (in
    # blocks of running sums, up to 1024 terms); the plan shows the passes,
    # the oracle the values
    w = wl.c5_vqe(B=8, n=n, layers=3, n_terms=n_terms)
    say("generated expectation passes n", n, "terms", n_terms)
    p = tq.Program(w.program_blob(), specialize=True)
    o = tq.Observables(w.observable_blob())
    th = dev(w.theta, torch.float32)
    e = tq.expectation(p, th, o).cpu().numpy()
    plan = tq.describe(p)
    ob = plan["groups"][0]["obs"]
    say("expectation passes", ob["exp_passes"], "H_g passes", ob["phi_passes"])
    assert sum(ob["exp_passes"]) == len(w.observables[0][0])
    ref = orc.expectation(orc.Program(w.program_blob()), w.theta.astype(np.float64), orc.Observables(w.observable_blob()))
    say("max |d exp|", float(np.abs(e - ref).max()))
    assert np.abs(e - ref).max() <= TOL_EXP * max(1.0, float(np.abs(ref).max()))
    # the table-driven Pauli kernel on the same inputs
    base = tq.expectation(tq.Program(w.program_blob()), th, o).cpu().numpy()
    assert np.abs(e - base).max() <= TOL_EXP


def test_specialized_bitwise_deterministic():
    # the generated kernels reduce in a fixed order too: two runs of the same
    # inputs agree bit for bit (forward passes, generated expectation and
    # H_g psi passes, reverse passes)
    for w in (wl.c5_vqe(B=16, n=14, layers=4, n_terms=120), wl.c3_qaoa(B=8, n=16)):
        a = gpu_outputs(w, want=("state", "exp", "grad"), specialize=True)
        b = gpu_outputs(w, want=("state", "exp", "grad"), specialize=True)
        for k in a:
            assert np.array_equal(a[k], b[k]), (w.name, k)
