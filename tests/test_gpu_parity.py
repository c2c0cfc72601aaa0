"""GPU parity: the HIP library against the complex128 oracle on the same
seeded inputs, at sizes the oracle finishes in seconds: random circuits over
the whole opcode set (heterogeneous batches, several tile passes, fixed bits,
partner tiles in HBM), planner options, determinism."""
import numpy as np
import pytest
import torch

from gpu_util import TOL_AMP, TOL_EXP, compare, dev, gpu_outputs, oracle_outputs, say
from oracle import oracle as orc
from paper_2003_02989_amd import tq
from paper_2003_02989_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", range(4))
def test_random_small_heterogeneous(seed):
    w = wl.random_batch(9000 + seed, B=6, n=7, n_gates=40, n_symbols=4, K=3, hetero=True)
    say("random small", seed)
    compare(gpu_outputs(w), oracle_outputs(w))


@pytest.mark.parametrize("n,tile,low", [(10, 8, 3), (12, 8, 6), (13, 9, 4), (14, 12, 6), (11, 8, 5)])
def test_random_tiled(n, tile, low):
    # n > tile: several passes, diagonal and control bits outside the tile,
    # expectation partners in other tiles
    w = wl.random_batch(100 * n + tile, B=3, n=n, n_gates=60, n_symbols=5, K=2)
    say("random tiled", n, tile, low)
    compare(gpu_outputs(w, max_tile_qubits=tile, low_qubits=low), oracle_outputs(w))


@pytest.mark.parametrize("n,tile,low", [(12, 8, 6), (14, 12, 6), (13, 9, 4)])
def test_specialized_passes_random(n, tile, low):
    # forward and reverse tile passes compiled for the circuit structure:
    # fixed bits, controls and diagonals outside the tile, dense stages
    w = wl.random_batch(100 * n + tile, B=3, n=n, n_gates=60, n_symbols=5, K=2)
    say("specialised passes", n, tile, low)
    compare(gpu_outputs(w, max_tile_qubits=tile, low_qubits=low, specialize=True), oracle_outputs(w))


def test_unfused_matches():
    w = wl.random_batch(4242, B=4, n=9, n_gates=50, n_symbols=3, K=2)
    compare(gpu_outputs(w, fuse=False), oracle_outputs(w))
    compare(gpu_outputs(w, max_tile_qubits=8, fuse=False), oracle_outputs(w))


def test_amplitudes_and_padding():
    w = wl.random_batch(77, B=5, n=8, n_gates=30, n_symbols=2, K=1, hetero=True)
    p = tq.Program(w.program_blob())
    th = dev(w.theta)
    st = tq.simulate_state(p, th).cpu().numpy()
    ref = oracle_outputs(w, want=("state",))["state"]
    for b, c in enumerate(w.circuits):
        assert not np.any(st[b, 1 << c.n:]), "zero padding"
    rng = np.random.default_rng(5)
    bits = np.stack([rng.integers(0, 1 << c.n, size=33) for c in w.circuits]).astype(np.int64)
    bits[0, 0] = 1 << 40  # out of range -> zero amplitude
    a = tq.amplitudes(p, th, dev(bits, torch.int64)).cpu().numpy()
    for b in range(w.B):
        for m in range(33):
            x = int(bits[b, m])
            want = ref[b, x] if x < ref.shape[1] and (x >> w.circuits[b].n) == 0 else 0
            assert abs(a[b, m] - want) < TOL_AMP


def test_bitwise_deterministic():
    w = wl.random_batch(31337, B=4, n=13, n_gates=60, n_symbols=6, K=3)
    a = gpu_outputs(w, max_tile_qubits=9)
    b = gpu_outputs(w, max_tile_qubits=9)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_no_symbols_and_empty_circuits():
    from paper_2003_02989_amd.circuits import Circuit
    c0 = Circuit(3)
    c1 = Circuit(2).add("H", 0).add("CNOT", (0, 1))
    w = wl.Workload("mixed", [c0, c1], 0, np.zeros((2, 0), np.float32),
                    [[[(1.0, [(0, "Z")]), (0.5, [])]], [[(1.0, [(0, "Z"), (1, "Z")])]]], np.ones((2, 1), np.float32))
    g = gpu_outputs(w, want=("state", "exp"))
    compare(g, oracle_outputs(w, want=("state", "exp")))
    assert abs(g["exp"][0, 0] - 1.5) < TOL_EXP and abs(g["exp"][1, 0] - 1.0) < TOL_EXP


@pytest.mark.parametrize("n", [3, 6, 12, 17])
def test_sampler_bit_exact_on_shared_state(n):
    rng = np.random.default_rng(n)
    B = 3
    z = (rng.standard_normal((B, 1 << n)) + 1j * rng.standard_normal((B, 1 << n))).astype(np.complex64)
    z /= np.linalg.norm(z, axis=1, keepdims=True)
    z = z.astype(np.complex64)
    z[1, ::3] = 0  # zero-probability outcomes are never drawn
    shots = 20000
    g = tq.sample_from_state(dev(z, torch.complex64), shots, seed=1234 + n).cpu().numpy().astype(np.uint64)
    r = orc.sample_from_state(z, shots, seed=1234 + n)
    say("sampler", n, "mismatches", int((g != r).sum()))
    assert np.array_equal(g, r)
    assert not np.any((g[1] % 3) == 0)


def test_full_pipeline_samples_fall_in_oracle_intervals():
    # samples of the complex64 pipeline must fall in the oracle's CDF interval
    # widened by the state difference (the two states differ by rounding)
    w = wl.random_batch(555, B=2, n=8, n_gates=40, n_symbols=3, K=1)
    p = tq.Program(w.program_blob())
    shots, seed = 4000, 99
    g = tq.sample(p, dev(w.theta), shots, seed).cpu().numpy().astype(np.uint64)
    ref_state = oracle_outputs(w, want=("state",))["state"]
    gst = tq.simulate_state(p, dev(w.theta)).cpu().numpy()
    for b in range(w.B):
        pr = np.abs(ref_state[b]) ** 2
        C = np.concatenate([[0.0], np.cumsum(pr)])
        delta = 2 * np.linalg.norm(gst[b] - ref_state[b]) + 1e-9
        for k in range(shots):
            u = orc.splitmix64(seed, b * shots + k) / 2.0 ** 64
            i = int(g[b, k])
            assert C[i] - delta <= u * C[-1] <= C[i + 1] + delta


@pytest.mark.parametrize("n,tile", [(14, 12), (9, 8), (6, 12)])
def test_many_observables_and_terms(n, tile):
    # K = 9 observables (three accumulation chunks), one of them an empty sum,
    # dense terms whose Z factors spread over the thread and register bits of
    # the Pauli tiles, X/Y factors outside the tile (partner tiles)
    rng = wl.rng_for(7000 + n)
    w = wl.random_batch(7100 + n, B=3, n=n, n_gates=50, n_symbols=4, K=9)
    for b in range(w.B):
        w.observables[b] = wl.random_observables(rng, n, 9, max_terms=14)
        w.observables[b][4] = []
    say("many observables", n, tile)
    compare(gpu_outputs(w, max_tile_qubits=tile), oracle_outputs(w))


def _z_observables(rng, n, K, many):
    # Z-only sums: one with `many` terms (more classes than one sweep of the
    # diagonal kernel holds), an empty one, identity terms, a repeated
    # string, and sum_i Z_i
    row = []
    for k in range(K):
        if k == 1:
            row.append([])
            continue
        if k == K - 1:
            row.append([(0.3, [(q, "Z")]) for q in range(n)])
            continue
        T = many if k == 0 else int(rng.integers(1, 6))
        terms = []
        for _ in range(T):
            w = int(rng.integers(0, 6))
            support = sorted(int(q) for q in rng.choice(n, size=w, replace=False)) if w else []
            terms.append((0.25 * float(rng.standard_normal()), [(q, "Z") for q in support]))
        if k == 2:
            terms += [terms[-1], (0.5, [])]
        row.append(terms)
    return row


@pytest.mark.parametrize("n,B,uniform", [(12, 3, False), (13, 2, False), (17, 2, False), (14, 4, True)])
def test_diagonal_observables(n, B, uniform):
    # Z-only observables on states of >= 12 qubits take the streaming
    # diagonal kernel (expectations) and the tile kernel (adjoint)
    rng = wl.rng_for(5100 + n)
    w = wl.random_batch(5200 + n, B=B, n=n, n_gates=50, n_symbols=4, K=5)
    shared = _z_observables(rng, n, 5, many=45)
    for b in range(B):
        w.observables[b] = shared if uniform else _z_observables(rng, n, 5, many=45)
    say("diagonal observables", n, B, uniform)
    compare(gpu_outputs(w), oracle_outputs(w))


@pytest.mark.parametrize("n,B", [(13, 3), (16, 2), (18, 2), (20, 1)])
def test_specialized_pauli_passes(n, B):
    # an observable set the same on every row (X/Y/Z strings of weight <= 4,
    # identity and Z-only terms, three observables) on states larger than a
    # tile: expectations by the passes compiled for it, each tile holding the
    # X bits of its terms
    rng = wl.rng_for(5300 + n)
    w = wl.random_batch(5400 + n, B=B, n=n, n_gates=60, n_symbols=4, K=3)
    shared = wl.random_observables(rng, n, 3, max_terms=12, max_weight=4)
    shared[1] = shared[1] + [(0.7, []), (-0.4, [(0, "Z"), (n - 1, "Z")])]
    for b in range(B):
        w.observables[b] = shared
    say("specialised Pauli passes", n, B)
    compare(gpu_outputs(w, want=("exp",), specialize=True), oracle_outputs(w, want=("exp",)))


@pytest.mark.parametrize("n,K,max_terms", [(15, 16, 60), (14, 2, 400), (14, 45, 8), (13, 200, 1)])
def test_specialized_pauli_passes_many(n, K, max_terms):
    # the generated expectation passes with their terms in several blocks:
    # sixteen observables (one accumulator each), two observables of a few
    # hundred terms (groups split across blocks), and more than sixteen
    # observables (sets of sixteen, each with passes of its own; 200
    # single-term observables as the sampled expectations' term values)
    w = wl.random_batch(5500 + n, B=2, n=n, n_gates=60, n_symbols=4, K=K)
    shared = wl.random_observables(wl.rng_for(5600 + n), n, K, max_terms=max_terms, max_weight=5)
    for b in range(w.B):
        w.observables[b] = shared
    say("specialised Pauli passes", n, "K", K, "terms", sum(len(o) for o in shared))
    p = tq.Program(w.program_blob(), specialize=True)
    e = tq.expectation(p, dev(w.theta), tq.Observables(w.observable_blob())).cpu().numpy()
    ob = tq.describe(p)["groups"][0]["obs"]
    say("generated expectation passes (terms per pass)", ob["exp_passes"], "sets", ob["exp_sets"])
    assert sum(ob["exp_passes"]) == sum(len(o) for o in shared)
    assert ob["exp_sets"] == (1 if K <= 16 else (K + 199) // 200)
    compare({"exp": e}, oracle_outputs(w, want=("exp",)))


@pytest.mark.gpu
def test_amplitudes_from_state_matches_amplitudes():
    # the state-based lookup returns what tq_amplitudes returns, bit for bit,
    # including out-of-range bitstrings (zero amplitude)
    w = wl.random_batch(4711, B=3, n=11, n_gates=40, n_symbols=3, K=1)
    p = tq.Program(w.program_blob())
    th = dev(w.theta)
    rng = np.random.default_rng(5)
    bits = rng.integers(0, 1 << 12, size=(3, 300)).astype(np.int64)
    b = torch.as_tensor(bits, device="cuda")
    st = tq.simulate_state(p, th)
    a1 = tq.amplitudes(p, th, b).cpu().numpy()
    a2 = tq.amplitudes_from_state(st, b).cpu().numpy()
    assert np.array_equal(a1, a2)
    assert np.all(a2[bits >= (1 << 11)] == 0)


@pytest.mark.parametrize("n,B", [(3, 5), (6, 9), (10, 7), (11, 3), (12, 2)])
def test_resident_layouts(n, B):
    # one wavefront per row (n <= 10; B not a multiple of the four rows of a
    # workgroup) and one workgroup per row (n = 11, 12)
    w = wl.random_batch(8800 + n, B=B, n=n, n_gates=70, n_symbols=6, K=2)
    say("resident", n, B)
    compare(gpu_outputs(w), oracle_outputs(w))


@pytest.mark.parametrize("seed", range(3))
def test_specialized_resident_random(seed):
    # structure-specialised resident kernels on heterogeneous batches of
    # random circuits over the whole opcode set (one kernel per structure),
    # states included (forward-only launches)
    w = wl.random_batch(6600 + seed, B=4, n=9 + seed, n_gates=60, n_symbols=5, K=3, hetero=True)
    say("specialised resident", seed)
    compare(gpu_outputs(w, specialize=True), oracle_outputs(w))


@pytest.mark.parametrize("n,max_terms,seed", [(13, 40, 0), (15, 150, 1)])
def test_specialized_hphi(n, max_terms, seed):
    # phi = g H psi from the kernels generated for one observable that is the
    # same on every row: partners across the tile's high bits, Y phases,
    # Z-only and identity terms, several passes
    w = wl.random_batch(7100 + seed, B=3, n=n, n_gates=50, n_symbols=5, K=1)
    obs = wl.random_observables(wl.rng_for(7200 + seed), n, 1, max_terms=max_terms, max_weight=4)
    w.observables = [obs for _ in range(w.B)]
    say("specialised H_g", n, len(obs[0]))
    compare(gpu_outputs(w, specialize=True), oracle_outputs(w))


def test_specialized_group_without_symbols():
    # adjoint over a batch whose first structure has no symbolic parameter
    # (no generated reverse passes: it takes the precompiled ones) next to one
    # with symbols, both run as tile passes
    w = wl.random_batch(7300, B=2, n=13, n_gates=40, n_symbols=3, K=2)
    w.circuits[0] = wl.random_circuit(wl.rng_for(7301), 13, 40, 3, p_symbolic=0.0)
    say("specialised group without symbols")
    compare(gpu_outputs(w, max_tile_qubits=10, specialize=True), oracle_outputs(w))


@pytest.mark.parametrize("specialize", [False, True])
@pytest.mark.parametrize("n,tile", [(2, 0), (13, 10)])
def test_yy_power_gradient(specialize, n, tile):
    # Y⊗Y^t built without its global phase: the adjoint gradient through it
    # (derivative matrices in the precompiled kernels, the gate's generator in
    # the generated ones), resident (n = 2) and in tile passes (n = 13,
    # 10-bit tiles), against the oracle
    from paper_2003_02989_amd.circuits import Circuit, sym
    c = Circuit(n).add("H", 0).add("RX", 1, [sym(1)]).add("YYPOW", (0, n - 1), [sym(0)])
    c.add("CNOT", (n - 1, 0)).add("YYPOW", (1, 0), [sym(0, 0.5, 0.1)])
    obs = [[(1.0, [(0, "Z")]), (0.5, [(0, "X"), (n - 1, "X")]), (-0.7, [(1, "Y")]), (0.3, [(0, "Y"), (1, "Y")])]]
    th = np.array([[0.37, 0.3], [-1.1, 2.0]], np.float32)
    w = wl.Workload("yy", [c, c], 2, th, [obs, obs], np.array([[1.0], [-0.6]], np.float32))
    say("YY^t gradient n", n, "specialize", specialize)
    compare(gpu_outputs(w, max_tile_qubits=tile, specialize=specialize), oracle_outputs(w))


def test_sampler_zero_row_marker():
    # a row without weight yields 2^64 - 1 for every shot on both sides; the
    # other rows are drawn as usual, bit-exact with the oracle
    rng = np.random.default_rng(4)
    z = (rng.standard_normal((3, 1 << 9)) + 1j * rng.standard_normal((3, 1 << 9))).astype(np.complex64)
    z /= np.linalg.norm(z, axis=1, keepdims=True)
    z = z.astype(np.complex64)
    z[1] = 0
    g = tq.sample_from_state(dev(z, torch.complex64), 3000, seed=8).cpu().numpy().astype(np.uint64)
    r = orc.sample_from_state(z, 3000, seed=8)
    assert np.all(g[1] == np.uint64(2**64 - 1))
    assert np.array_equal(g, r)


@pytest.mark.parametrize("specialize", [False, True])
@pytest.mark.parametrize("n,seed", [(9, 0), (13, 1), (15, 2)])
def test_pauli_exponentials_random(n, seed, specialize):
    # Pauli-string exponentials of every weight (0 to n, X/Y/Z letters,
    # symbolic with shared symbols, or constant) interleaved with random
    # gates: states, expectations and adjoint gradients against the oracle
    # (resident states, and tile passes of 13 and 15 qubits)
    from paper_2003_02989_amd.circuits import Circuit, const, sym
    rng = wl.rng_for(8100 + seed)
    w = wl.random_batch(8200 + seed, B=3, n=n, n_gates=30, n_symbols=4, K=2)
    for c in w.circuits:
        for _ in range(8):
            wt = int(rng.integers(0, n + 1))
            fac = [(int(q), "XYZ"[int(rng.integers(0, 3))]) for q in rng.choice(n, size=wt, replace=False)]
            par = (sym(int(rng.integers(0, 4)), float(rng.normal()), float(rng.normal())) if rng.random() < 0.75
                   else const(float(rng.normal())))
            e = Circuit(n).add_pauli_exp(fac, par).gates[0]
            c.gates.insert(int(rng.integers(0, len(c.gates) + 1)), e)
    say("Pauli exponentials", n, seed, "specialize", specialize)
    compare(gpu_outputs(w, specialize=specialize), oracle_outputs(w))


@pytest.mark.parametrize("specialize", [False, True])
@pytest.mark.parametrize("n,seed", [(8, 0), (13, 1)])
def test_noisy_trajectories(n, seed, specialize):
    # Pauli channels (depolarizing after every gate, plus asymmetric ones):
    # every row a trajectory whose Paulis are drawn from the noise seed; the
    # draws are bit-exact between the two sides, so states, expectations and
    # adjoint gradients match the oracle row by row; tq_row_mean averages the
    # trajectories of each circuit
    from paper_2003_02989_amd.circuits import Circuit
    base = wl.random_batch(8300 + seed, B=2, n=n, n_gates=25, n_symbols=3, K=2)
    for c in base.circuits:
        c.add("PCHAN", 0, [0.2, 0.05, 0.3])
        c.add("PCHAN", n - 1, [0.0, 0.0, 0.5])
    R = 6
    w = wl.with_noise(base, 0.08, R)
    for noise_seed in (11, 12):
        say("noisy trajectories n", n, "seed", noise_seed, "specialize", specialize)
        orc.set_noise_seed(noise_seed)
        orc.set_row_offset(0)
        p = tq.Program(w.program_blob(), specialize=specialize)
        tq.set_noise_seed(p, noise_seed)
        o = tq.Observables(w.observable_blob())
        th = dev(w.theta)
        st = tq.simulate_state(p, th).cpu().numpy()
        e = tq.expectation(p, th, o)
        ge = torch.empty((w.B, w.K), dtype=torch.float32, device="cuda")
        g = tq.adjoint_grad(p, th, o, dev(w.upstream), expectations=ge).cpu().numpy()
        compare({"state": st, "exp": e.cpu().numpy(), "grad": g, "grad_exp": ge.cpu().numpy()}, oracle_outputs(w))
        m = tq.row_mean(e, R).cpu().numpy()
        assert np.abs(m - e.cpu().numpy().reshape(base.B, R, w.K).astype(np.float64).mean(1)).max() < 1e-6
    # the trajectories differ from row to row (the noise is applied)
    assert np.abs(st[0] - st[1]).max() > 1e-3 or np.abs(st[1] - st[2]).max() > 1e-3


@pytest.mark.parametrize("n,seed", [(14, 0), (18, 1)])
def test_phase_classes(n, seed):
    # ZZ-type layers that the generated passes apply as phase classes (one
    # table lookup of w^cut per amplitude): RZZ on a random graph with one
    # symbol, ZZ^t with another symbol and scale, RZZ with a constant angle,
    # and a ZZ^t layer whose symbols differ per edge (no class); states,
    # expectations, adjoint and parameter-shift gradients against the oracle
    from paper_2003_02989_amd.circuits import Circuit, const, observable_blob, program_blob, sym
    rng = np.random.default_rng(4400 + seed)
    edges = wl.random_regular3(rng, n)
    dense = sorted({(int(a), int(b)) for a, b in (sorted(rng.choice(n, 2, replace=False)) for _ in range(3 * n))})
    c = Circuit(n)
    for q in range(n):
        c.add("H", q)
    for a, b in edges:
        c.add("RZZ", (a, b), [sym(0)])
    for q in range(n):
        c.add("RX", q, [sym(1)])
    for a, b in dense:
        c.add("ZZPOW", (a, b), [sym(2, -0.7, 0.1)])
    for a, b in edges:
        c.add("RZZ", (a, b), [const(0.37)])
    for q in range(n):
        c.add("RY", q, [sym(3)])
    for i, (a, b) in enumerate(edges):
        c.add("ZZPOW", (a, b), [sym(4 + i % 3)])
    for q in range(0, n, 2):
        c.add("RX", q, [sym(1)])
    B, S = 3, 7
    theta = rng.uniform(-3, 3, size=(B, S)).astype(np.float32)
    obs = [[[(0.5, [(a, "Z"), (b, "Z")]) for a, b in edges[:6]] + [(0.3, [(0, "X"), (n - 1, "Y")])]]] * B
    from paper_2003_02989_amd.workloads import Workload
    w = Workload("phase_classes", [c] * B, S, theta, obs, rng.standard_normal((B, 1)).astype(np.float32))
    say("phase classes n", n, "edges", len(edges), "dense", len(dense))
    compare(gpu_outputs(w, specialize=True), oracle_outputs(w))
    p = tq.Program(w.program_blob(), specialize=True)
    o = tq.Observables(w.observable_blob())
    g = tq.param_shift_grad(p, dev(w.theta), o, dev(w.upstream)).cpu().numpy()
    ref = orc.param_shift_grad(orc.Program(w.program_blob()), w.theta.astype(np.float64),
                               orc.Observables(w.observable_blob()), w.upstream.astype(np.float64))
    say("  parameter-shift error", float(np.abs(g - ref).max()))
    assert np.abs(g - ref).max() <= 1e-4
