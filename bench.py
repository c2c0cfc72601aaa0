"""Benchmark of the batched state-vector hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config c4|c1|c2|c3|c5] [--expectation-only]
                    [--no-cpu-baseline]

One step is one call of the configuration's hot path on its full batch with
inputs resident in HBM and a new parameter set (or sampling seed) per step:
  c4  tq_sample_with_amplitudes: one simulation of the 30-qubit random circuit
      (40 fused tile passes over the 8 GiB state), its amplitudes at 4096
      bitstrings and 10^6 samples (the default workload)
  c1, c2, c5  tq_adjoint_grad with expectation output (forward passes, Pauli-sum
              expectations, H_g, reverse adjoint passes, gradient reduction);
              with --expectation-only tq_expectation
  c3  tq_expectation
Rank 0 prints one JSON line.  `value` is the metric's half that fits the
workload: for c4 the effective HBM GB/s of its fused-gate passes
(16 B per amplitude per pass, 8 B for the pass that generates the product
state, over the passes' HIP-event time); for the batched workloads
circuit-expectations/s over the step time.  Both figures, the cold start
(library load + program creation + first call, in two fresh processes: one
with an empty code-object cache, which compiles every generated kernel, one
with the cache the first filled) and the dominant kernel's HBM and fp64
rooflines are in the line; the oracle, timed on the host's cores on a bounded
sample, gives the cpu_baseline entry.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective HBM GB/s per fused-gate pass; circuit-expectations/sec at batch"
KERNELS = ("build", "resident", "pass", "pauli", "pauli_reduce", "rev_pass", "grad_reduce", "sampled_counts",
           "samp_l1", "samp_shots", "gather")
MODELLED = ("resident", "pass", "pauli", "rev_pass")
PEAK_HBM_GBS = 8000.0
PEAK_FP64_TFLOPS = 78.6  # fp64 vector: 256 CUs x 2.4 GHz x 128 flop/clk


# HBM traffic per launch of a dominant kernel, from rocprofv3 FETCH_SIZE and
# WRITE_SIZE runs (profiles/traffic.json, scaled by the counters' reading for
# a plain device copy of known size).  Valid only for the sources it was
# measured with: the hash below must match.
TRAFFIC_SOURCES = tuple("paper_2003_02989_amd/csrc/" + f for f in (
    "kernels.hip", "kernels.h", "kernel_args.h", "device_ops.h", "tq_internal.h", "program.cpp", "program.h",
    "tq_abi.cpp", "jit.cpp", "jit.h"))


def sources_hash():
    import hashlib
    h = hashlib.sha256()
    root = os.path.dirname(os.path.abspath(__file__))
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(root, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(config, kernel):
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("sources_sha256") != sources_hash():
        return None
    e = t.get("configs", {}).get(config)
    if not e or e.get("kernel") != kernel:
        return None
    return e.get("bytes_per_launch")


def workload(name):
    from paper_2003_02989_amd import workloads as wl
    return wl.CONFIGS[name]()


def describe_workload(name, w, adjoint=True, mode="plain", reps=0, eps=0.0):
    d = describe_config(name, w, w.B // w.extras.get("trajectories", 1))
    if mode == "sampled":
        d = d.replace("expectations+adjoint grads", "expectations") + f", sampled expectations ({reps} shots per term)"
    elif mode == "param-shift":
        d = d.replace("expectations+adjoint grads", "expectations") + ", parameter-shift gradients" + (
            f" from sampled expectations ({reps} shots per term)" if reps else "")
    elif mode == "finite-diff":
        d = d.replace("expectations+adjoint grads", "expectations") + f", central-difference gradients (eps {eps})"
    if "trajectories" in w.extras:
        d += (f", depolarizing noise p={w.extras['noise_p']} after every gate, "
              f"{w.extras['trajectories']} trajectories per circuit (B={w.B} trajectory rows)")
    if name in ("c1", "c2", "c5") and not adjoint and mode == "plain":
        d = d.replace("expectations+adjoint grads", "expectations only")
    return d


def describe_config(name, w, B):
    n = w.n_max
    if name == "c1":
        return f"c1 hardware-efficient ansatz n={n} B={B} 2 layers RX,RY,RZ + CZ ladder, sum Z, expectations+adjoint grads"
    if name == "c2":
        return f"c2 QNN classifier n={n} B={B} RX(pi x) encoding + 4 layers ZZ^t, XX^t to readout, Z_9, expectations+adjoint grads"
    if name == "c3":
        how = " layers from Pauli-string exponentials of H_C, H_M," if w.name.startswith("c3_qaoa_exp") else ""
        return f"c3 QAOA MaxCut n={n} B={B} p=4 random 3-regular graph,{how} cut observable, expectations"
    if name == "c4":
        return f"c4 random circuit n={n} B=1 depth 20 sqrtX/Y/W + fSim 5x6 grid, 4096 amplitudes + 10^6 samples"
    return f"c5 VQE ansatz n={n} B={B} 10 layers RY,RZ + CNOT ring, 200 Pauli strings, expectations+adjoint grads"


# Algorithmic work of one op applied to one amplitude, in the form the plan
# gives the op (its structure hints, PassOp::hint): complex mul = 6 flops,
# complex add = 2, a real times a complex = 2.  2x2: dense 14, real or
# "RX form" (real diagonal, imaginary off-diagonal) 6, exactly X 0; a
# controlled 2x2 touches half the amplitudes.  Diagonal: 6 per entry that is
# not exactly 1, over the entries' share of amplitudes.  Excitation
# preserving (fSim-like): the |00>, |11> phases that are not 1 (6 on a quarter
# each) and the (|01>, |10>) block on half (dense 14, RX form 6, -i SWAP 0).
# Pauli pair 14 (6 in RX form), dense 4x4 30.  Constant single-qubit gates
# the generated kernels write out with unit entries folded (sqrt X: 2) are
# still counted by their hint, so the count is an upper bound of the
# arithmetic done.
H_X, H_REAL, H_RX, H_SWAP = 16, 32, 64, 128


def op_flops(op, n_local_ctrl):
    k, h = op["kind"], op.get("hint", 0)
    if k == "M1":
        f = 0.0 if h & H_X else 6.0 if h & (H_REAL | H_RX) else 14.0
        return f / 2 if (op["ctrl"] and n_local_ctrl) else f
    if k == "M2":
        return 30.0
    if k == "P2":
        return 6.0 if h & H_RX else 14.0
    if k == "F2":
        ph = 1.5 * ((0 if h & 1 else 1) + (0 if h & 8 else 1))
        blk = 0.0 if h & H_SWAP else 3.0 if h & H_RX else 7.0
        return ph + blk
    # diagonal: D1 has 2 entries (half the amplitudes each), D2 4 (a quarter)
    units = bin(h & (3 if k == "D1" else 15)).count("1")
    n_ent = 2 if k == "D1" else 4
    return 6.0 * (n_ent - units) / n_ent


def fwd_flops(g):
    f = 0.0
    for i, ps in enumerate(g["fwd"]):
        f += 12.0 if ps["product_init"] else 0.0
        for op in ps["ops"]:
            f += op_flops(op, op["ctrl"] and op["l"][1] != 255)
    return f


def rev_flops(g):
    f = 0.0
    for ps in g["rev"]:
        for op in ps["ops"]:
            base = op_flops(op, op["ctrl"] and op["l"][1] != 255)
            f += 2 * base + op["ngrad"] * (base + 4.0)
    return f


def kernel_work(plan, kernel, n_obs_terms, adjoint):
    """Algorithmic (flops, HBM bytes) of all launches of `kernel` in one step,
    and the number of those launches, from the program's plan.  Per amplitude:
    a forward op costs its matvec (op_flops), a reverse op two matvecs (psi
    and phi) plus one matvec and a 4-flop dot product per symbolic parameter,
    an expectation term 4 flops, an H_g term 4 more."""
    flops = bytes_ = 0.0
    launches = 0
    for g in plan["groups"]:
        amps = float(g["rows"]) * (1 << g["n"])
        if kernel == "resident":
            launches += 1
            f = fwd_flops(g) + 4.0 * n_obs_terms
            if adjoint:
                f += 8.0 * n_obs_terms + rev_flops(g)
            flops += f * amps
            bytes_ += 0.0
        elif kernel == "pass":
            for ps in g["fwd"]:
                launches += 1
                f = 12.0 if ps["product_init"] else 0.0
                for op in ps["ops"]:
                    f += op_flops(op, op["ctrl"] and op["l"][1] != 255)
                flops += f * amps
                bytes_ += (8.0 if ps["product_init"] else 16.0) * amps
        elif kernel == "rev_pass":
            for i, ps in enumerate(g["rev"]):
                launches += 1
                f = 0.0
                for op in ps["ops"]:
                    base = op_flops(op, op["ctrl"] and op["l"][1] != 255)
                    f += 2 * base + op["ngrad"] * (base + 4.0)
                flops += f * amps
                bytes_ += (32.0 if i + 1 < len(g["rev"]) else 16.0) * amps
        elif kernel == "pauli":
            # expectations: 4 flops per term and amplitude, psi read; with the
            # adjoint also phi = H_g psi (4 more, phi written, and read back by
            # every pass after the first).  The generated passes split the
            # terms over several launches (the plan's "obs" entry).
            ob = g.get("obs", {})
            passes = ob.get("phi_passes") if adjoint else (ob.get("exp_passes") or ob.get("phi_passes"))
            if passes and not (ob.get("diag") and not adjoint):
                for i, nt in enumerate(passes):
                    launches += 1
                    flops += (8.0 if adjoint else 4.0) * nt * amps
                    bytes_ += ((16.0 if i == 0 else 24.0) if adjoint else 8.0) * amps
            else:
                launches += 1
                flops += (8.0 if adjoint else 4.0) * n_obs_terms * amps
                bytes_ += (16.0 if adjoint else 8.0) * amps
    return flops, bytes_, launches


def expansion(plan, w, mode):
    """Rows the step runs per row of the batch: 1, or for the shift rules the
    shifted circuits (2 per symbolic blob parameter; central differences: 2
    per symbol a row uses), averaged over the batch."""
    if mode == "param-shift":
        tot = sum(g["rows"] * 2 * len(g["occurrences"]) for g in plan["groups"])
    elif mode == "finite-diff":
        tot = 0
        for c in w.circuits:
            used = {p[0] for _, _, params, _ in c.gates for p in params if p[0] >= 0}
            tot += 2 * len(used)
    else:
        return 1.0
    return tot / max(w.B, 1)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def progress(msg):
    """One line per finished phase on stderr (the JSON line is the only
    stdout output)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c4", choices=["c1", "c2", "c3", "c4", "c5"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--expectation-only", action="store_true",
                    help="c1, c2, c5: time tq_expectation (no adjoint gradients)")
    ap.add_argument("--noise", type=float, default=0.0,
                    help="c1, c2, c3, c5: depolarizing channel of this probability after every gate on its qubits, "
                         "simulated as --trajectories trajectories per circuit (averaged)")
    ap.add_argument("--trajectories", type=int, default=10)
    ap.add_argument("--pauli-exp", action="store_true",
                    help="c3: the QAOA layers built from Pauli-string exponentials of the cost and mixer "
                         "Hamiltonians")
    ap.add_argument("--mode", default="plain", choices=["plain", "sampled", "param-shift", "finite-diff"],
                    help="c1, c2, c3, c5: plain = adjoint gradients (c1, c2, c5) or expectations (c3); "
                         "sampled = tq_sampled_expectation with --reps shots per term; param-shift = "
                         "tq_param_shift_grad (--reps > 0: from sampled expectations); finite-diff = "
                         "tq_finite_diff_grad with step --eps")
    ap.add_argument("--reps", type=int, default=None,
                    help="shots per term (sampled: default 1000; param-shift: default 0 = exact)")
    ap.add_argument("--eps", type=float, default=1e-2)
    ap.add_argument("--no-specialize", action="store_true",
                    help="run with the precompiled table-driven kernels instead of the ones compiled for the "
                         "circuit structure on the first call")
    ap.add_argument("--low-qubits", type=int, default=0,
                    help="contiguous low index bits of every tile (0: the library's default)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the workload step: HBM sweep of single-gate passes and expectation kernels")
    ap.add_argument("--sweep-cases", default="all", choices=["all", "gates", "expectation"],
                    help="with --sweep: which kernels to sweep")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the two cold-start child runs (empty, then filled code-object cache)")
    ap.add_argument("--cold-probe", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy a 1 GiB device buffer three times (reference for the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has no multi-GPU mode; "
              "the batch would split across GPUs row-wise and a large state by amplitudes",
              file=sys.stderr)
        sys.exit(1)

    # cold start in fresh processes before this one touches the GPU: library
    # load, program creation and first call with an empty code-object cache
    # (every generated kernel compiled), then again with the cache it filled
    cold = None
    cache_tmp = None
    if not (args.sweep or args.copy_calibration or args.cold_probe or args.no_cold or args.no_specialize):
        import shutil
        import subprocess
        import tempfile
        cache_tmp = tempfile.mkdtemp(prefix="tq-bench-cache-")
        env = dict(os.environ, TQ_CACHE_DIR=cache_tmp)
        cmd = [sys.executable, os.path.abspath(__file__), "--cold-probe", "--config", args.config]
        if args.expectation_only:
            cmd.append("--expectation-only")
        if args.pauli_exp:
            cmd.append("--pauli-exp")
        if args.noise > 0:
            cmd += ["--noise", str(args.noise), "--trajectories", str(args.trajectories)]
        cmd += ["--mode", args.mode, "--eps", str(args.eps)]
        if args.reps is not None:
            cmd += ["--reps", str(args.reps)]
        cold = {}
        for key in ("empty_cache", "filled_cache"):
            r = subprocess.run(cmd, env=env, capture_output=True, text=True, timeout=900)
            if r.returncode != 0:
                print(r.stdout[-2000:], r.stderr[-4000:], file=sys.stderr)
                sys.exit(r.returncode)
            cold[key] = json.loads(r.stdout.strip().splitlines()[-1])
            progress(f"cold start ({key.replace('_', ' ')}) {cold[key]['cold_ms']:.0f} ms")
        os.environ["TQ_CACHE_DIR"] = cache_tmp

    import numpy as np
    import torch

    from paper_2003_02989_amd import tq
    from paper_2003_02989_amd import workloads as wl

    local_rank = int(os.environ.get("LOCAL_RANK", "0"))
    torch.cuda.set_device(local_rank)
    if args.sweep:
        sweep(args.steps, args.sweep_cases, not args.no_specialize)
        return
    if args.copy_calibration:
        src = torch.ones(1 << 27, dtype=torch.complex64, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": 8 << 27, "bytes_written": 8 << 27, "copies": 3}))
        return
    if args.pauli_exp and args.config != "c3":
        print("--pauli-exp applies to c3 only", file=sys.stderr)
        sys.exit(1)
    w = wl.c3_qaoa(exponentials=True) if args.pauli_exp else workload(args.config)
    noisy = args.noise > 0
    mode = args.mode
    if mode != "plain" and (args.config == "c4" or args.expectation_only):
        print("--mode applies to c1, c2, c3, c5 (without --expectation-only)", file=sys.stderr)
        sys.exit(1)
    reps = args.reps if args.reps is not None else (1000 if mode == "sampled" else 0)
    if noisy and args.config == "c4":
        print("--noise applies to c1, c2, c3, c5", file=sys.stderr)
        sys.exit(1)
    R = args.trajectories if noisy else 1
    w_base = w
    if noisy:
        w = wl.with_noise(w_base, args.noise, R)
    B, K = w.B, w.K
    adjoint = args.config in ("c1", "c2", "c5") and not args.expectation_only and mode == "plain"
    specialize = not args.no_specialize
    # every step (first call, warm-up, per-kernel profiling, timed) gets its
    # own parameter set, drawn like the workload's
    prof_steps = 1 if mode in ("param-shift", "finite-diff") else 2
    n_prof = prof_steps * len(KERNELS)
    n_steps_total = 1 + args.warmup + n_prof + args.steps
    # (the trajectories of a noisy circuit share its parameters)
    thetas = ([torch.as_tensor(np.repeat(t, R, axis=0), device="cuda")
               for t in wl.fresh_thetas(w_base, n_steps_total, 7 + wl.BASE_SEED)]
              if w.n_symbols else [None] * n_steps_total)
    up = torch.as_tensor(w.upstream, device="cuda")
    exp = torch.empty((B, K), dtype=torch.float32, device="cuda")
    grad = torch.empty((B, w.n_symbols), dtype=torch.float32, device="cuda")
    exp_mean = torch.empty((B // R, K), dtype=torch.float32, device="cuda")
    grad_mean = torch.empty((B // R, w.n_symbols), dtype=torch.float32, device="cuda")
    if args.config == "c4":
        bits = torch.as_tensor(w.extras["bitstrings"].astype(np.int64), device="cuda")
        amps = torch.empty((1, bits.shape[1]), dtype=torch.complex64, device="cuda")
        n_shots = w.extras["n_shots"]
        shots = torch.empty((1, n_shots), dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()

    counter = [0]

    def step():
        i = counter[0]
        counter[0] += 1
        th = thetas[i]
        if noisy:  # new trajectories every step
            tq.set_noise_seed(prog, 1000 + i)
        if mode == "sampled":
            tq.sampled_expectation(prog, th, obs, reps, 5000 + i, out=exp)
            if noisy:
                tq.row_mean(exp, R, out=exp_mean)
        elif mode in ("param-shift", "finite-diff"):
            if mode == "param-shift":
                tq.param_shift_grad(prog, th, obs, up, reps=reps, seed=5000 + i, grad=grad)
            else:
                tq.finite_diff_grad(prog, th, obs, up, args.eps, grad=grad)
            if noisy:
                tq.row_mean(grad, R, out=grad_mean)
        elif adjoint:
            tq.adjoint_grad(prog, th, obs, up, grad=grad, expectations=exp)
            if noisy:
                tq.row_mean(grad, R, out=grad_mean)
                tq.row_mean(exp, R, out=exp_mean)
        elif args.config != "c4":
            tq.expectation(prog, th, obs, out=exp)
            if noisy:
                tq.row_mean(exp, R, out=exp_mean)
        else:
            # one simulation serves both outputs; a new sampling seed per step
            tq.sample_with_amplitudes(prog, None, n_shots, w.extras["seed"] + i, bits, out=shots, amps=amps)

    # cold: library loaded, program and observables created, first call
    # (kernels generated for the structure, compiled or read from the code
    # cache)
    # (the serialised inputs are built beforehand: they are the caller's)
    pblob, oblob = w.program_blob(), w.observable_blob()
    t0 = time.perf_counter()
    tq.lib()
    t_load = time.perf_counter() - t0
    t0 = time.perf_counter()
    prog = tq.Program(pblob, specialize=specialize, low_qubits=args.low_qubits)
    obs = tq.Observables(oblob)
    t_create = time.perf_counter() - t0
    t0 = time.perf_counter()
    step()
    torch.cuda.synchronize()
    t_first = time.perf_counter() - t0
    if args.cold_probe:
        print(json.dumps({"load_ms": t_load * 1e3, "create_ms": t_create * 1e3, "first_call_ms": t_first * 1e3,
                          "cold_ms": (t_load + t_create + t_first) * 1e3}), flush=True)
        return
    progress(f"first call {t_first * 1e3:.0f} ms")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    progress("warm-up done")

    # dominant kernel: device time per step of every kernel, from HIP events
    per_kernel = {}
    for kname in KERNELS:
        tq.profile_start(kname)
        for _ in range(prof_steps):
            step()
        torch.cuda.synchronize()
        n_l, ms = tq.profile_read()
        tq.profile_start(None)
        if n_l:
            per_kernel[kname] = ms / prof_steps
            progress(f"kernel {kname}: {ms / prof_steps:.3f} ms per step")
    # (among the kernels of the simulation and expectation path, whose work
    # kernel_work models; the builder's small matrices and the samplers are
    # reported in kernel_ms_per_step only)
    dominant = max((k for k in per_kernel if k in MODELLED), key=per_kernel.get)

    # timed region; the dominant kernel's launches are bracketed by events
    tq.profile_start(dominant)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    n_launch, dom_ms = tq.profile_read()
    tq.profile_start(None)
    ms_per_step = elapsed * 1e3 / args.steps
    progress(f"timed {args.steps} steps: {ms_per_step:.3f} ms per step")

    plan = tq.describe(prog)
    n_terms = sum(len(t) for t in w.observables[0])
    flops, bytes_, launches_per_step = kernel_work(plan, dominant, n_terms, adjoint)
    # the shift rules run every row's shifted circuits (derived rows) through
    # the same kernels: the work of a plain step times the rows per row
    expand = expansion(plan, w, mode)
    flops *= expand
    bytes_ *= expand
    if mode in ("param-shift", "finite-diff"):  # launches are per chunk of derived rows: count them
        launches_per_step = n_launch / args.steps
    avg_ms = dom_ms / max(n_launch, 1)
    # (the stored counters are per workload: noisy rows, shift-rule expansions
    # and sampled modes launch other sizes and have entries of their own)
    traffic = measured_traffic(args.config + ("_expectation" if args.expectation_only else "")
                               + ("_pauli_exp" if args.pauli_exp else "")
                               + (f"_noisy{R}" if noisy else "")
                               + ("" if mode == "plain" else "_" + mode), dominant)
    per_launch_flops = flops / max(launches_per_step, 1)
    per_launch_bytes = bytes_ / max(launches_per_step, 1)
    hbm = {"bound": "hbm", "achieved": per_launch_bytes / (avg_ms * 1e-3) / 1e9, "peak": PEAK_HBM_GBS,
           "unit": "GB/s", "algorithmic_per_launch": per_launch_bytes}
    hbm["frac"] = hbm["achieved"] / hbm["peak"]
    alu = {"bound": "alu", "achieved": per_launch_flops / (avg_ms * 1e-3) / 1e12, "peak": PEAK_FP64_TFLOPS,
           "unit": "TFLOP/s", "algorithmic_per_launch": per_launch_flops, "arithmetic": "fp64 vector"}
    alu["frac"] = alu["achieved"] / alu["peak"]
    binding, other = (hbm, alu) if hbm["frac"] >= alu["frac"] else (alu, hbm)
    roofline = dict(binding)
    roofline.update({"kernel": dominant, "traffic": traffic, "launches_per_step": launches_per_step,
                     "avg_launch_ms": avg_ms, "other_roof": other})

    # the two halves of the metric
    pass_bytes = kernel_work(plan, "pass", n_terms, adjoint)[1] * expand
    if dominant == "pass":
        pass_ms = dom_ms / args.steps
    else:
        pass_ms = per_kernel.get("pass", 0.0)
    fused_pass_gbs = pass_bytes / (pass_ms * 1e-3) / 1e9 if pass_ms > 0 else None
    # cold start: the fresh process with an empty code cache when it ran,
    # else this process (library load, creation, first call)
    here = {"load_ms": t_load * 1e3, "create_ms": t_create * 1e3, "first_call_ms": t_first * 1e3,
            "cold_ms": (t_load + t_create + t_first) * 1e3}
    cold_s = (cold["empty_cache"] if cold else here)["cold_ms"] * 1e-3
    cached_s = cold["filled_cache"]["cold_ms"] * 1e-3 if cold else None
    if args.config == "c4":
        value, unit_v = fused_pass_gbs, "GB/s (effective HBM bandwidth per fused-gate pass)"
        rates = {"amplitudes_per_s": B * amps.shape[1] / (ms_per_step * 1e-3),
                 "samples_per_s": B * n_shots / (ms_per_step * 1e-3),
                 "fused_passes_per_step": kernel_work(plan, "pass", n_terms, adjoint)[2],
                 "fused_pass_ms_per_step": pass_ms,
                 "cold_ms": cold_s * 1e3,
                 "cold_cached_ms": cached_s * 1e3 if cached_s else None}
    else:
        # noisy: one circuit-expectation is the mean over its R trajectories
        Bc = B // R
        value = Bc * K / (ms_per_step * 1e-3)
        unit_v = "circuit-expectations/s" + (" (with adjoint gradients)" if adjoint else "")
        if mode == "sampled":
            unit_v = f"circuit-expectations/s (sampled, {reps} shots per term)"
        if mode in ("param-shift", "finite-diff"):
            value = Bc / (ms_per_step * 1e-3)
            unit_v = ("gradient rows/s (" + ("parameter shift" if mode == "param-shift" else
                                             f"central differences, eps {args.eps}")
                      + f", {expand:g} shifted circuits per row" + (f", {reps} shots per term" if reps else "") + ")")
        if noisy:
            unit_v += f" (noisy: mean of {R} trajectories each)"
        rates = {"circuit_expectations_per_s": Bc * K / (ms_per_step * 1e-3),
                 "cold_circuit_expectations_per_s": Bc * K / cold_s,
                 "cold_cached_circuit_expectations_per_s": Bc * K / cached_s if cached_s else None,
                 "fused_pass_GBps": fused_pass_gbs,
                 "fused_pass_ms_per_step": pass_ms if pass_ms > 0 else None}
        if mode in ("param-shift", "finite-diff"):
            rates["gradient_rows_per_s"] = value
            rates["shifted_circuits_per_step"] = expand * B
            rates["shifted_circuit_expectations_per_s"] = expand * B * K / (ms_per_step * 1e-3)
        if noisy:
            rates["trajectory_rows_per_s"] = B / (ms_per_step * 1e-3)
        if adjoint:
            rates["gradient_rows_per_s"] = Bc / (ms_per_step * 1e-3)

    line = {
        "metric": METRIC,
        "value": value,
        "unit": unit_v,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic (seeded generators, no datasets); a new parameter set or sampling seed per step",
        "config": {"workload": describe_workload(args.config, w, adjoint, mode, reps, args.eps), "storage": "complex64",
                   "arithmetic": "fp64",
                   "batch": B, "qubits": w.n_max, "symbols": w.n_symbols, "observables": K,
                   "pauli_terms": n_terms, "specialized_kernel": specialize,
                   "noise": {"depolarizing_p": args.noise, "trajectories": R} if noisy else None},
        "cold_start": {"fresh_process_empty_code_cache": cold["empty_cache"] if cold else None,
                       "fresh_process_filled_code_cache": cold["filled_cache"] if cold else None,
                       "this_process": here},
        "rates": rates,
        "roofline": roofline,
        "kernel_ms_per_step": per_kernel,
    }

    if not args.no_cpu_baseline and local_rank == 0:
        line["cpu_baseline"] = cpu_baseline(args.config, w, args.cpu_seconds, adjoint, R, mode, reps, args.eps)
    print(json.dumps(line), flush=True)
    if cache_tmp:
        shutil.rmtree(cache_tmp, ignore_errors=True)


def sweep(steps, cases="all", specialize=True):
    """Effective HBM bandwidth of single-gate passes and of the expectation
    kernel for n = 24..30 with batches sized so the states span >= 1 GiB (the
    256 MB last-level cache cannot hold them).  A pass time is the difference
    of two programs with max_pass_gates = 1 (every gate its own pass) that
    differ by G test gates (or G fused blocks of gates, max_pass_gates = the
    block's size), divided by the difference of their pass counts.  One JSON
    line per case."""
    import numpy as np
    import torch

    from paper_2003_02989_amd import tq
    from paper_2003_02989_amd.circuits import Circuit, const, observable_blob, program_blob
    from paper_2003_02989_amd.workloads import random_unitary

    G = 8
    tile = int(os.environ.get("TQ_SWEEP_TILE", "0"))
    low = int(os.environ.get("TQ_SWEEP_LOW", "0"))

    # plain device copy of the same footprint: the practical HBM ceiling
    for n in ((26, 30) if cases in ("all", "gates") else ()):
        B = max(1, (1 << 27) >> n)
        src = torch.empty((B, 1 << n), dtype=torch.complex64, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        gbs = 16.0 * (1 << n) * B / (ms * 1e-3) / 1e9
        print(json.dumps({"sweep": "device_copy", "n": n, "batch": B, "case": "torch copy_", "ms": ms,
                          "GB_per_s": gbs, "frac_of_8TBps": gbs / PEAK_HBM_GBS}), flush=True)
        del src, dst

    def pass_ms(n, B, prefix, gate, block=None):
        # block: the test gates as a list applied G times, with max_pass_gates
        # equal to its length, so that each test pass applies one block's
        # worth of gates on its qubits, fused
        block = block or [gate]
        times, passes = [], []
        for with_test in (True, False):
            circuits = []
            for _ in range(B):
                c = Circuit(n)
                for g in prefix:
                    c.add(*g)
                if with_test:
                    for _ in range(G):
                        for g in block:
                            c.add(*g)
                circuits.append(c)
            prog = tq.Program(program_blob(circuits, 0), max_tile_qubits=tile, low_qubits=low,
                              max_pass_gates=len(block), specialize=specialize)
            passes.append(sum(len(g["fwd"]) for g in tq.describe(prog)["groups"]))
            st = torch.empty((B, 1 << n), dtype=torch.complex64, device="cuda")
            tq.simulate_state(prog, None, out=st)
            torch.cuda.synchronize()
            tq.profile_start("pass")
            for _ in range(steps):
                tq.simulate_state(prog, None, out=st)
            torch.cuda.synchronize()
            nl, ms = tq.profile_read()
            tq.profile_start(None)
            times.append(ms / steps)
            del st, prog
        return (times[0] - times[1]) / (passes[0] - passes[1])

    for n in (24, 26, 28, 30):
        B = max(1, (1 << 27) >> n)
        q = lambda bit: n - 1 - bit  # qubit on index bit `bit`
        gate_cases = []
        for bit in sorted({0, 3, 6, 10, n - 1}):
            gate_cases.append((f"1q RX on bit {bit}", [("CZ", (q(bit), q((bit + 1) % n)))], ("RX", q(bit), [const(0.3)])))
        gate_cases.append((f"fSim on bits {n-1},{n-2}", [("CZ", (q(n - 1), q(n - 2)))],
                      ("FSIM", (q(n - 1), q(n - 2)), [const(0.7), const(0.4)])))
        gate_cases.append(("fSim on bits 0,1", [("CZ", (q(0), q(1)))], ("FSIM", (q(0), q(1)), [const(0.7), const(0.4)])))
        gate_cases.append((f"XX^t on bits {n-1},{n-2}", [("CZ", (q(n - 1), q(n - 2)))],
                      ("XXPOW", (q(n - 1), q(n - 2)), [const(0.3)])))
        gate_cases.append((f"CNOT control bit {n-1}, target bit 0", [("CZ", (q(n - 1), q(0)))], ("CNOT", (q(n - 1), q(0)))))
        gate_cases.append((f"RZZ on bits {n-1},0 (diagonal)", [("CZ", (q(n - 1), q(0)))], ("RZZ", (q(n - 1), q(0)), [const(0.3)])))
        # fused k-qubit windows on the top bits: a random unitary on each of
        # the k qubits and on each neighbouring pair (2k - 1 dense gates, one
        # pass per block)
        urng = np.random.default_rng(1000 + n)
        for k in (2, 3, 4, 5):
            qs = [q(n - 1 - j) for j in range(k)]
            blk = [("MATRIX1", qs[j], [], random_unitary(urng, 2)) for j in range(k)]
            blk += [("MATRIX2", (qs[j], qs[j + 1]), [], random_unitary(urng, 4)) for j in range(k - 1)]
            gate_cases.append((f"fused k={k} window on bits {n-1}..{n-k} ({2 * k - 1} dense gates)",
                               [("CZ", (qs[0], qs[1]))], None, blk))
        for case in (gate_cases if cases in ("all", "gates") else []):
            name, prefix, gate = case[:3]
            ms = pass_ms(n, B, prefix, gate, case[3] if len(case) > 3 else None)
            gbs = 16.0 * (1 << n) * B / (ms * 1e-3) / 1e9
            print(json.dumps({"sweep": "gate_pass", "n": n, "batch": B, "case": name, "ms_per_pass": ms,
                              "GB_per_s": gbs, "frac_of_8TBps": gbs / PEAK_HBM_GBS}), flush=True)
        if cases not in ("all", "expectation"):
            continue
        # expectation kernels on a product state (RY, RZ on every qubit: one
        # fused pass) whose expectations have a closed form, checked on every
        # row: sum_i Z_i, 30 random Z_i Z_j plus a constant (the QAOA cost's
        # shape), 16 random X/Y/Z strings, 200 (the VQE Hamiltonian's shape)
        # and sixteen observables of 650 strings over all
        from paper_2003_02989_amd.workloads import random_pauli_strings
        rng = np.random.default_rng(n)
        obs_sets = {"sum Z_i": [[(1.0, [(i, "Z")]) for i in range(n)]],
                    "16 XYZ strings": [[(float(rng.standard_normal()),
                                         [(int(x), "XYZ"[int(rng.integers(0, 3))])
                                          for x in rng.choice(n, size=int(rng.integers(1, 5)), replace=False)])
                                        for _ in range(16)]],
                    "30 ZZ + constant": [[(-0.5, [(int(a), "Z"), (int(b), "Z")])
                                          for a, b in (rng.choice(n, size=2, replace=False) for _ in range(30))]
                                         + [(15.0, [])]],
                    "200 XYZ strings": [random_pauli_strings(rng, n, 200)],
                    "16 observables, 650 strings": [random_pauli_strings(rng, n, 200)]
                    + [random_pauli_strings(rng, n, 30) for _ in range(15)]}
        ang_t = rng.uniform(0.0, 2 * np.pi, size=n)
        ang_f = rng.uniform(0.0, 2 * np.pi, size=n)
        c = Circuit(n)
        for i in range(n):
            c.add("RY", i, [const(float(ang_t[i]))])
            c.add("RZ", i, [const(float(ang_f[i]))])
        comp = [{"X": np.sin(ang_t[q]) * np.cos(ang_f[q]), "Y": np.sin(ang_t[q]) * np.sin(ang_f[q]),
                 "Z": np.cos(ang_t[q])} for q in range(n)]
        prog = tq.Program(program_blob([c] * B, 0), specialize=specialize)
        for oname, sums in obs_sets.items():
            K = len(sums)
            obs = tq.Observables(observable_blob([sums] * B))
            out = torch.empty((B, K), dtype=torch.float32, device="cuda")
            tq.expectation(prog, None, obs, out=out)
            torch.cuda.synchronize()
            ref = np.array([sum(cf * np.prod([comp[q][p] for q, p in fac]) for cf, fac in terms) for terms in sums])
            err = float(np.abs(out.cpu().numpy() - ref[None, :]).max())
            tol = float((1e-6 * np.array([sum(abs(cf) for cf, _ in t) for t in sums]) + 1e-6).min())
            tq.profile_start("pauli")
            for _ in range(steps):
                tq.expectation(prog, None, obs, out=out)
            torch.cuda.synchronize()
            nl, ms = tq.profile_read()
            tq.profile_start(None)
            ms /= steps  # every launch of the call (one per pass of the plan)
            n_terms = sum(len(t) for t in sums)
            gbs = 8.0 * (1 << n) * B / (ms * 1e-3) / 1e9
            tfs = 4.0 * n_terms * (1 << n) * B / (ms * 1e-3) / 1e12
            print(json.dumps({"sweep": "expectation", "n": n, "batch": B, "case": oname, "terms": n_terms,
                              "ms": ms, "launches_per_call": nl // steps,
                              "GB_per_s": gbs, "frac_of_8TBps": gbs / PEAK_HBM_GBS,
                              "fp64_TFLOP_per_s": tfs, "frac_of_fp64_peak": tfs / PEAK_FP64_TFLOPS,
                              "closed_form_max_error": err, "closed_form_ok": err <= tol}), flush=True)
        del prog


def cpu_baseline(name, w, budget_s, adjoint=True, R=1, mode="plain", reps=0, eps=1e-2):
    """The oracle on the host cores, on a bounded sample of the same workload."""
    import numpy as np

    from oracle import oracle as orc
    orc.build()
    threads = orc.num_threads()
    if name == "c4":
        from paper_2003_02989_amd import workloads as wl
        ws = wl.c4_random(rows=4, cols=6, n_shots=10_000)
        p = orc.Program(ws.program_blob())
        t0 = time.perf_counter()
        reps = 0
        while True:
            orc.amplitudes(p, np.zeros((1, 0)), ws.extras["bitstrings"])
            reps += 1
            if time.perf_counter() - t0 > budget_s:
                break
        dt = (time.perf_counter() - t0) / reps
        # the metric's unit: 16 B per amplitude per gate application of the
        # oracle's gate-by-gate sweeps (it applies every gate as its own pass)
        n_g = len(ws.circuits[0].gates)
        gbs = 16.0 * (1 << ws.circuits[0].n) * n_g / dt / 1e9
        return {"value": gbs, "unit": "GB/s (effective, 16 B per amplitude per gate pass)", "cores": threads,
                "kind": "oracle", "cpu": cpu_model(), "amplitudes_per_s": 4096 / dt,
                "sample": f"24-qubit stand-in (4x6 grid) of the depth-20 random circuit, {n_g} gates, one full "
                          f"complex128 simulation plus 4096 amplitudes per call, {reps} calls in {dt * reps:.1f} s"}
    if mode in ("param-shift", "finite-diff"):
        # the oracle simulates every shifted circuit in full: one row costs
        # `expand` expectation evaluations.  Rows are timed directly when one
        # fits the budget; otherwise the expectation of sampled rows is timed
        # and scaled by the shifted circuits per row (what the oracle's
        # shift rule runs for each row).
        from paper_2003_02989_amd.workloads import Workload
        sub = Workload(w.name, [w.circuits[0]], w.n_symbols, w.theta[:1], [w.observables[0]], w.upstream[:1])
        p = orc.Program(sub.program_blob())
        o = orc.Observables(sub.observable_blob())
        th = sub.theta.astype(np.float64)
        t0 = time.perf_counter()
        orc.expectation(p, th, o)
        t_exp = time.perf_counter() - t0
        n_shift = 2 * (sum(1 for _, _, params, _ in w.circuits[0].gates for q in params if q[0] >= 0)
                       if mode == "param-shift" else
                       len({q[0] for _, _, params, _ in w.circuits[0].gates for q in params if q[0] >= 0}))
        if t_exp * n_shift > budget_s:
            n_e = 1
            t0 = time.perf_counter()
            while time.perf_counter() - t0 < budget_s:
                orc.expectation(p, th, o)
                n_e += 1
            dt = (time.perf_counter() - t0 + t_exp) / n_e
            return {"value": 1.0 / (dt * n_shift) / R, "unit": "gradient rows/s", "cores": threads,
                    "kind": "oracle", "cpu": cpu_model(),
                    "sample": f"{n_e} complex128 expectation evaluations of row 0 in {dt * n_e:.1f} s, scaled by the "
                              f"{n_shift} shifted circuits the oracle's "
                              + ("parameter-shift" if mode == "param-shift" else "central-difference")
                              + " rule simulates per row"}
    rows = 1
    done_rows = 0
    t0 = time.perf_counter()
    while True:
        r = list(range(min(rows, w.B)))
        from paper_2003_02989_amd.workloads import Workload
        sub = Workload(w.name, [w.circuits[i] for i in r], w.n_symbols, w.theta[r], [w.observables[i] for i in r],
                       w.upstream[r])
        p = orc.Program(sub.program_blob())
        o = orc.Observables(sub.observable_blob())
        th = sub.theta.astype(np.float64)
        if mode == "sampled":
            orc.sampled_expectation(p, th, o, reps, 1)
        elif mode == "param-shift":
            orc.param_shift_grad(p, th, o, sub.upstream.astype(np.float64), reps, 1)
        elif mode == "finite-diff":
            orc.finite_diff_grad(p, th, o, sub.upstream.astype(np.float64), eps)
        else:
            orc.expectation(p, th, o)
            if adjoint:
                orc.adjoint_grad(p, th, o, sub.upstream.astype(np.float64))
        done_rows += len(r)
        el = time.perf_counter() - t0
        if el > budget_s:
            break
        rows = min(max(rows * 2, 1), w.B)
    what = "expectations" + (" + adjoint gradients" if adjoint else "")
    if mode != "plain":
        what = {"sampled": f"sampled expectations, {reps} shots per term",
                "param-shift": "parameter-shift gradients" + (f" from {reps} shots per term" if reps else ""),
                "finite-diff": f"central-difference gradients, eps {eps}"}[mode]
    if mode in ("param-shift", "finite-diff"):
        return {"value": done_rows / R / el, "unit": "gradient rows/s", "cores": threads, "kind": "oracle",
                "cpu": cpu_model(),
                "sample": f"{done_rows} rows of the same batch ({what}, rows repeated in doubling chunks up to "
                          f"the full batch) in {el:.1f} s"}
    return {"value": done_rows / R * w.K / el, "unit": "circuit-expectations/s", "cores": threads, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{done_rows} rows of the same batch ({what}, rows repeated in doubling chunks up to "
                      f"the full batch) in {el:.1f} s"}


if __name__ == "__main__":
    main()
