"""Helpers of the GPU parity tests: run a workload through the HIP library
(via the binding) and through the oracle on the same seeded inputs."""
import sys

import numpy as np
import torch

from oracle import oracle as orc
from paper_2003_02989_amd import tq

TOL_EXP = 1e-5   # absolute, expectations (complex64 path)
TOL_GRAD = 1e-4  # absolute, gradients
TOL_AMP = 1e-5   # L2 error of a state / amplitude vector


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(x, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(x)).to(device="cuda", dtype=dtype)


def gpu_outputs(w, want=("state", "exp", "grad"), **opts):
    p = tq.Program(w.program_blob(), **opts)
    o = tq.Observables(w.observable_blob())
    th = dev(w.theta) if w.n_symbols else None
    out = {}
    if "state" in want:
        out["state"] = tq.simulate_state(p, th).cpu().numpy()
    if "exp" in want:
        out["exp"] = tq.expectation(p, th, o).cpu().numpy()
    if "grad" in want:
        e = torch.empty((w.B, w.K), dtype=torch.float32, device="cuda")
        g = tq.adjoint_grad(p, th, o, dev(w.upstream), expectations=e)
        out["grad"] = g.cpu().numpy()
        out["grad_exp"] = e.cpu().numpy()
    torch.cuda.synchronize()
    return out


def oracle_outputs(w, want=("state", "exp", "grad")):
    p = orc.Program(w.program_blob())
    o = orc.Observables(w.observable_blob())
    th = w.theta.astype(np.float64)
    out = {}
    if "state" in want:
        out["state"] = orc.simulate_state(p, th)
    if "exp" in want:
        out["exp"] = orc.expectation(p, th, o)
    if "grad" in want:
        out["grad"] = orc.adjoint_grad(p, th, o, w.upstream.astype(np.float64))
    return out


def compare(gpu, ref, tol_exp=TOL_EXP, tol_grad=TOL_GRAD, tol_amp=TOL_AMP):
    if "state" in ref:
        err = np.linalg.norm(gpu["state"].astype(np.complex128) - ref["state"], axis=1)
        assert err.max() <= tol_amp, f"state L2 error {err.max():.3e}"
    if "exp" in ref:
        err = np.abs(gpu["exp"] - ref["exp"]).max()
        assert err <= tol_exp, f"expectation error {err:.3e}"
    if "grad" in ref:
        err = np.abs(gpu["grad"] - ref["grad"]).max() if ref["grad"].size else 0.0
        assert err <= tol_grad, f"gradient error {err:.3e}"
        if "exp" in ref:
            err = np.abs(gpu["grad_exp"] - ref["exp"]).max()
            assert err <= tol_exp, f"expectation (adjoint call) error {err:.3e}"


def sub_workload(w, rows):
    """The rows `rows` of workload w as a workload of their own (the oracle
    computes sampled rows of a full-size batch one by one)."""
    from paper_2003_02989_amd.workloads import Workload
    rows = list(rows)
    return Workload(w.name + "_rows", [w.circuits[r] for r in rows], w.n_symbols, w.theta[rows],
                    [w.observables[r] for r in rows], w.upstream[rows], dict(w.extras))
