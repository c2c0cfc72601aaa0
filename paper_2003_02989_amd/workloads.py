"""Seeded synthetic workloads shaped like the paper's QML circuits.

Input generation only: random draws and circuit/observable construction, no
simulation arithmetic.  Both the HIP path and the oracle consume what these
functions emit (the blobs of ``circuits.py`` plus numpy arrays).

Every generator draws from ``numpy.random.Generator(PCG64(seed))`` in a fixed
order; the default seed of configuration c is 200302989 + c.  The five
configurations stand in for the paper's workloads (its datasets, Cirq's
supremacy-circuit generator, MNIST and the molecular data are not available):

  c1  hardware-efficient ansatz, 4 qubits, batch 16 (RL / PQC circuits,
      Sec. "Policy-Gradient Reinforcement Learning with PQCs")
  c2  10-qubit QNN classifier, batch 1024 (Sec. "Layerwise quantum circuit
      learning": data qubits coupled to a readout qubit by ZZ^t and XX^t)
  c3  QAOA MaxCut on a random 3-regular graph, 20 qubits, p=4, batch 256
      (Sec. "Quantum Approximate Optimization", scaled up from 10 nodes, p=1)
  c4  30-qubit random circuit of depth 20 on a 5x6 grid with sqrt(X),
      sqrt(Y), sqrt(W) and fSim(pi/2, pi/6) (the dense random circuits of
      Sec. "Benchmarks")
  c5  16-qubit VQE-style ansatz, 10 layers of RY, RZ and a CNOT ring, batch
      4096, 200 random Pauli strings of weight <= 4 (Sec. "Subspace-Search
      Variational Quantum Eigensolver")
"""
import math
from dataclasses import dataclass, field

import numpy as np

from .circuits import Circuit, const, observable_blob, program_blob, sym

BASE_SEED = 200302989


def rng_for(seed):
    return np.random.Generator(np.random.PCG64(seed))


@dataclass
class Workload:
    name: str
    circuits: list
    n_symbols: int
    theta: np.ndarray            # float32 [B, S]
    observables: list            # [B][K] list of terms
    upstream: np.ndarray         # float32 [B, K]
    extras: dict = field(default_factory=dict)

    @property
    def B(self):
        return len(self.circuits)

    @property
    def K(self):
        return len(self.observables[0]) if self.observables else 0

    @property
    def n_max(self):
        return max(c.n for c in self.circuits)

    def program_blob(self):
        return program_blob(self.circuits, self.n_symbols)

    def observable_blob(self):
        return observable_blob(self.observables)


def _repeat_obs(terms, B, K=1):
    return [[terms for _ in range(K)] for _ in range(B)]


# ----------------------------------------------------------------------- c1
def c1_hea(B=16, n=4, layers=2, seed=BASE_SEED + 1):
    """Per layer: RX, RY, RZ on every qubit (symbol index l*3n + 3q + axis),
    then the CZ ladder CZ(q_i, q_{i+1}).  Observable sum_i Z_i."""
    rng = rng_for(seed)
    S = layers * n * 3
    theta = rng.uniform(0.0, 2 * math.pi, size=(B, S)).astype(np.float32)
    c = Circuit(n)
    for l in range(layers):
        for q in range(n):
            for a, g in enumerate(("RX", "RY", "RZ")):
                c.add(g, q, [sym(l * 3 * n + 3 * q + a)])
        for q in range(n - 1):
            c.add("CZ", (q, q + 1))
    obs = [(1.0, [(q, "Z")]) for q in range(n)]
    return Workload("c1_hea", [c] * B, S, theta, _repeat_obs(obs, B), np.ones((B, 1), np.float32))


# ----------------------------------------------------------------------- c2
def c2_qnn(B=1024, n_data=9, layers=4, seed=BASE_SEED + 2):
    """Encoding RX(pi*x_i), x_i ~ U{0,1}, on the data qubits (per-row
    constants), then per layer ZZ(q_i, q_r)^theta for every data qubit and
    XX(q_i, q_r)^theta, readout qubit r = n_data; symbol l*2*n_data +
    kind*n_data + i.  The same symbol values on every row.  Observable Z_r."""
    rng = rng_for(seed)
    n = n_data + 1
    r = n_data
    x = rng.integers(0, 2, size=(B, n_data))
    S = layers * 2 * n_data
    th = rng.uniform(0.0, 2 * math.pi, size=S).astype(np.float32)
    theta = np.broadcast_to(th, (B, S)).copy()
    circuits = []
    for b in range(B):
        c = Circuit(n)
        for i in range(n_data):
            c.add("RX", i, [const(math.pi * float(x[b, i]))])
        for l in range(layers):
            for i in range(n_data):
                c.add("ZZPOW", (i, r), [sym(l * 2 * n_data + i)])
            for i in range(n_data):
                c.add("XXPOW", (i, r), [sym(l * 2 * n_data + n_data + i)])
        circuits.append(c)
    obs = [(1.0, [(r, "Z")])]
    return Workload("c2_qnn", circuits, S, theta, _repeat_obs(obs, B), np.ones((B, 1), np.float32),
                    {"x": x})


# ----------------------------------------------------------------------- c3
def random_regular3(rng, n):
    """Random 3-regular simple graph by the pairing (configuration) model with
    rejection: 3n half-edges, a uniformly random perfect matching, rejected
    while it has a loop or a repeated edge.  Edges sorted."""
    while True:
        half = np.repeat(np.arange(n), 3)
        perm = rng.permutation(half)
        pairs = perm.reshape(-1, 2)
        edges = set()
        ok = True
        for a, b in pairs:
            a, b = int(min(a, b)), int(max(a, b))
            if a == b or (a, b) in edges:
                ok = False
                break
            edges.add((a, b))
        if ok:
            return sorted(edges)


def c3_qaoa(B=256, n=20, p=4, seed=BASE_SEED + 3, exponentials=False):
    """H on every qubit, then per layer l: RZZ(gamma_l) on every edge and
    RX(beta_l) on every qubit; symbols gamma_1..p = 0..p-1, beta = p..2p-1,
    (gamma, beta) ~ U[0, pi).  Observable sum_edges 0.5 (1 - Z_i Z_j) =
    |E|/2 * I - 0.5 sum_edges Z_i Z_j.

    exponentials=True builds the layers as the paper's QAOA example does,
    from the exponentials of the two Hamiltonians: exp(-i gamma_l H_C) as the
    product of its terms' exponentials (the constant one a global phase, each
    -0.5 Z_i Z_j one Pauli-string exponential), then exp(-i beta_l sum X_i)
    as one exponential per qubit."""
    rng = rng_for(seed)
    edges = random_regular3(rng, n)
    theta = rng.uniform(0.0, math.pi, size=(B, 2 * p)).astype(np.float32)
    obs = [(0.5 * len(edges), [])] + [(-0.5, [(a, "Z"), (b, "Z")]) for a, b in edges]
    c = Circuit(n)
    for q in range(n):
        c.add("H", q)
    for l in range(p):
        if exponentials:
            for coeff, factors in obs:
                c.add_pauli_exp(factors, sym(l, coeff))
            for q in range(n):
                c.add_pauli_exp([(q, "X")], sym(p + l))
            continue
        for a, b in edges:
            c.add("RZZ", (a, b), [sym(l)])
        for q in range(n):
            c.add("RX", q, [sym(p + l)])
    return Workload("c3_qaoa_exp" if exponentials else "c3_qaoa", [c] * B, 2 * p, theta, _repeat_obs(obs, B),
                    np.ones((B, 1), np.float32), {"edges": edges})


# ----------------------------------------------------------------------- c4
def grid_couplers(rows, cols):
    """Couplers of a rows x cols grid, qubit (r, c) -> cols*r + c.  Pattern A:
    horizontal with c even, B: horizontal with c odd, C: vertical with r even,
    D: vertical with r odd.  Pairs are (lower index, higher index)."""
    pat = {"A": [], "B": [], "C": [], "D": []}
    for r in range(rows):
        for c in range(cols - 1):
            pat["A" if c % 2 == 0 else "B"].append((cols * r + c, cols * r + c + 1))
    for r in range(rows - 1):
        for c in range(cols):
            pat["C" if r % 2 == 0 else "D"].append((cols * r + c, cols * (r + 1) + c))
    return pat


def c4_random(rows=5, cols=6, depth=20, n_bitstrings=4096, n_shots=1_000_000, seed=BASE_SEED + 4):
    """Per cycle j: a random single-qubit gate from {sqrt(X), sqrt(Y),
    sqrt(W)} on every qubit (cycle 0 uniform over the three, later cycles
    uniform over the two that differ from the qubit's previous gate; draws in
    cycle order, then qubit order), then fSim(pi/2, pi/6) on the couplers of
    pattern "ABCD"[j mod 4].  Then n_bitstrings uniform bitstrings."""
    rng = rng_for(seed)
    n = rows * cols
    pat = grid_couplers(rows, cols)
    names = ("SQRTX", "SQRTY", "SQRTW")
    c = Circuit(n)
    prev = [None] * n
    for j in range(depth):
        for q in range(n):
            if prev[q] is None:
                g = int(rng.integers(0, 3))
            else:
                choices = [k for k in range(3) if k != prev[q]]
                g = choices[int(rng.integers(0, 2))]
            prev[q] = g
            c.add(names[g], q)
        for a, b in pat["ABCD"[j % 4]]:
            c.add("FSIM", (a, b), [const(math.pi / 2), const(math.pi / 6)])
    bitstrings = rng.integers(0, 1 << n, size=(1, n_bitstrings), dtype=np.uint64)
    theta = np.zeros((1, 0), np.float32)
    obs = [[[(1.0, [(0, "Z")])]]]
    return Workload(f"c4_random_n{n}", [c], 0, theta, obs, np.ones((1, 1), np.float32),
                    {"bitstrings": bitstrings, "n_shots": n_shots, "seed": seed})


# ----------------------------------------------------------------------- c5
def random_pauli_strings(rng, n, count, max_weight=4):
    """Weight w ~ U{1..max_weight}, support of w distinct uniform qubits,
    each factor uniform in {X, Y, Z}, coefficient ~ N(0, 1); duplicates of an
    earlier string are drawn again until `count` distinct strings exist."""
    seen = set()
    terms = []
    while len(terms) < count:
        w = int(rng.integers(1, max_weight + 1))
        support = sorted(int(q) for q in rng.choice(n, size=w, replace=False))
        paulis = [("X", "Y", "Z")[int(rng.integers(0, 3))] for _ in range(w)]
        coeff = float(rng.standard_normal())
        key = tuple(zip(support, paulis))
        if key in seen:
            continue
        seen.add(key)
        terms.append((coeff, list(key)))
    return terms


def c5_vqe(B=4096, n=16, layers=10, n_terms=200, seed=BASE_SEED + 5):
    """Per layer l: RY, RZ on every qubit (symbols l*2n + 2q + {0, 1}), then
    CNOT(q_i, q_{(i+1) mod n}) for i ascending.  Hamiltonian: n_terms random
    Pauli strings (drawn first), then theta ~ U[0, 2 pi)."""
    rng = rng_for(seed)
    terms = random_pauli_strings(rng, n, n_terms)
    S = layers * 2 * n
    theta = rng.uniform(0.0, 2 * math.pi, size=(B, S)).astype(np.float32)
    c = Circuit(n)
    for l in range(layers):
        for q in range(n):
            c.add("RY", q, [sym(l * 2 * n + 2 * q)])
            c.add("RZ", q, [sym(l * 2 * n + 2 * q + 1)])
        for i in range(n):
            c.add("CNOT", (i, (i + 1) % n))
    return Workload("c5_vqe", [c] * B, S, theta, _repeat_obs(terms, B), np.ones((B, 1), np.float32))


# ------------------------------------------------------------ random tests
ONE_Q = ["H", "X", "Y", "Z", "RX", "RY", "RZ", "XPOW", "YPOW", "ZPOW", "SQRTX", "SQRTY", "SQRTW", "MATRIX1"]
TWO_Q = ["CZ", "CNOT", "CZPOW", "CNOTPOW", "XXPOW", "YYPOW", "ZZPOW", "RZZ", "FSIM", "MATRIX2", "SWAP"]


def random_unitary(rng, d):
    z = rng.standard_normal((d, d)) + 1j * rng.standard_normal((d, d))
    q, r = np.linalg.qr(z)
    return q * (np.diag(r) / np.abs(np.diag(r)))


def random_circuit(rng, n, n_gates, n_symbols, p_symbolic=0.6, ops=None):
    """A random circuit over the whole opcode set; parameters are symbolic
    with probability p_symbolic (random symbol, scale in [-2, 2], offset in
    [-1, 1]) and constants otherwise.  ``Circuit.gates`` holds the plain
    (name, qubits, params, matrix) tuples."""
    from .circuits import OPS
    c = Circuit(n)
    pool = list(ops) if ops is not None else (ONE_Q + (TWO_Q if n >= 2 else []))
    for _ in range(n_gates):
        name = pool[int(rng.integers(0, len(pool)))]
        _, nq, npar = OPS[name]
        qubits = tuple(int(q) for q in rng.choice(n, size=nq, replace=False))
        params = []
        for _ in range(npar):
            if n_symbols > 0 and rng.random() < p_symbolic:
                params.append(sym(int(rng.integers(0, n_symbols)), float(rng.uniform(-2, 2)),
                                  float(rng.uniform(-1, 1))))
            else:
                params.append(const(float(rng.uniform(-math.pi, math.pi))))
        matrix = None
        if name == "MATRIX1":
            matrix = random_unitary(rng, 2)
        elif name == "MATRIX2":
            matrix = random_unitary(rng, 4)
        c.add(name, qubits, params, matrix)
    return c


def random_observables(rng, n, K, max_terms=5, max_weight=None):
    row = []
    for _ in range(K):
        T = int(rng.integers(1, max_terms + 1))
        terms = []
        for _ in range(T):
            w = int(rng.integers(0, (max_weight or n) + 1))
            support = sorted(int(q) for q in rng.choice(n, size=w, replace=False)) if w else []
            terms.append((float(rng.standard_normal()), [(q, ("X", "Y", "Z")[int(rng.integers(0, 3))]) for q in support]))
        row.append(terms)
    return row


def random_batch(seed, B, n, n_gates, n_symbols, K=2, hetero=False, **kw):
    """A batch of B random circuits (different structures) and observables."""
    rng = rng_for(seed)
    circuits, obs = [], []
    for b in range(B):
        nb = int(rng.integers(1, n + 1)) if hetero else n
        circuits.append(random_circuit(rng, nb, n_gates, n_symbols, **kw))
        obs.append(random_observables(rng, nb, K))
    theta = rng.uniform(-math.pi, math.pi, size=(B, n_symbols)).astype(np.float32)
    upstream = rng.standard_normal((B, K)).astype(np.float32)
    return Workload(f"random_n{n}", circuits, n_symbols, theta, obs, upstream)


def with_noise(w, p, R):
    """The noisy version of workload w as trajectories: after every gate a
    depolarizing channel of probability p on each qubit the gate acts on (the
    paper's circuit-wide depolarizing model: the channel after each
    operation, Sec. "Training Models with Noise"), and every row repeated R
    times (rows b R .. b R + R - 1 are the trajectories of circuit b; their
    outputs average with tq_row_mean)."""
    circuits, memo = [], {}
    for c in w.circuits:
        nc = memo.get(id(c))  # one noisy circuit per distinct circuit object
        if nc is None:
            nc = memo[id(c)] = Circuit(c.n)
            for g in c.gates:
                nc.gates.append(g)
                for q in g[1]:
                    nc.depolarize(q, p)
        circuits += [nc] * R
    rep = lambda a: np.repeat(a, R, axis=0)
    return Workload(w.name + f"_noisy{R}", circuits, w.n_symbols, rep(w.theta),
                    [o for o in w.observables for _ in range(R)], rep(w.upstream),
                    dict(w.extras, noise_p=p, trajectories=R))


CONFIGS = {"c1": c1_hea, "c2": c2_qnn, "c3": c3_qaoa, "c4": c4_random, "c5": c5_vqe}


def fresh_thetas(w, count, seed):
    """`count` further symbol-value arrays [B, S] drawn like the workload's
    own: U[0, pi) for the QAOA angles, one shared U[0, 2 pi) row for the QNN,
    U[0, 2 pi) per entry otherwise (a new parameter set per benchmark step)."""
    rng = rng_for(seed)
    out = []
    for _ in range(count):
        if w.name.startswith("c3"):
            th = rng.uniform(0.0, math.pi, size=w.theta.shape)
        elif w.name.startswith("c2"):
            th = np.broadcast_to(rng.uniform(0.0, 2 * math.pi, size=w.theta.shape[1]), w.theta.shape)
        else:
            th = rng.uniform(0.0, 2 * math.pi, size=w.theta.shape)
        out.append(np.ascontiguousarray(th, dtype=np.float32))
    return out
