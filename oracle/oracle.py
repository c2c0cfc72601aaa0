"""ctypes wrapper of the complex128 CPU oracle (``liboracle.so``).

TEST INFRASTRUCTURE ONLY: imported by tests/, ``__graft_entry__.smoke()`` and
the cpu_baseline leg of bench.py, never by the product package.

Inputs are program / observable blobs (bytes) and numpy arrays; outputs are
numpy arrays.  Symbol values are taken as float64 (callers that compare with
the float32 GPU path pass the same float32 values widened exactly).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# TQ_ORACLE_LIB: another build of the same source (the sanitizer test loads one)
_LIB_PATH = os.environ.get("TQ_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "tq_oracle.c")


def build(force=False):
    """Compile the oracle with gcc (plain C11 + OpenMP)."""
    if not force and os.path.exists(_LIB_PATH) and os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    cmd = ["gcc", "-O2", "-std=gnu11", "-fopenmp", "-fPIC", "-shared", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    subprocess.check_call(cmd)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        vp, sz, i32, i64, u64 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64
        dp = ctypes.POINTER(ctypes.c_double)
        L.orc_last_error.restype = ctypes.c_char_p
        L.orc_program_parse.argtypes = [ctypes.c_char_p, sz, ctypes.POINTER(vp)]
        L.orc_program_free.argtypes = [vp]
        L.orc_program_info.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(i32), vp]
        L.orc_obs_parse.argtypes = [ctypes.c_char_p, sz, ctypes.POINTER(vp)]
        L.orc_obs_free.argtypes = [vp]
        L.orc_simulate_state.argtypes = [vp, vp, vp]
        L.orc_expectation.argtypes = [vp, vp, vp, vp, vp]
        L.orc_adjoint_grad.argtypes = [vp, vp, vp, vp, vp]
        L.orc_amplitudes.argtypes = [vp, vp, vp, i64, vp]
        L.orc_sample.argtypes = [vp, vp, i64, u64, vp]
        L.orc_sample_from_state.argtypes = [vp, i32, i32, i64, u64, vp]
        L.orc_gate_matrix.argtypes = [i32, vp, vp, vp, ctypes.POINTER(i32)]
        L.orc_gate_dmatrix.argtypes = [i32, vp, i32, vp, ctypes.POINTER(i32)]
        L.orc_splitmix64.argtypes = [u64, u64]
        L.orc_splitmix64.restype = u64
        L.orc_set_c64_storage.argtypes = [i32]
        L.orc_num_threads.restype = i32
        L.orc_op_arity.argtypes = [i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.orc_set_noise_seed.argtypes = [u64]
        L.orc_set_row_offset.argtypes = [i64]
        L.orc_sampled_expectation.argtypes = [vp, vp, vp, i32, u64, vp]
        L.orc_sampled_from_terms.argtypes = [vp, vp, i32, i32, u64, vp]
        L.orc_channel_pick.argtypes = [u64, i64, i32, ctypes.c_double, ctypes.c_double, ctypes.c_double]
        L.orc_channel_pick.restype = i32
        L.orc_param_shift_grad.argtypes = [vp, vp, vp, vp, i32, u64, vp]
        L.orc_finite_diff_grad.argtypes = [vp, vp, vp, vp, ctypes.c_double, vp]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc):
    if rc != 0:
        raise OracleError(lib().orc_last_error().decode())


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


class Program:
    def __init__(self, blob: bytes):
        h = ctypes.c_void_p()
        _check(lib().orc_program_parse(blob, len(blob), ctypes.byref(h)))
        self._h = h
        B, S, nmax = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        lib().orc_program_info(h, ctypes.byref(B), ctypes.byref(S), ctypes.byref(nmax), None)
        self.B, self.S, self.nmax = B.value, S.value, nmax.value
        nq = np.zeros(self.B, dtype=np.int32)
        lib().orc_program_info(h, ctypes.byref(B), ctypes.byref(S), ctypes.byref(nmax), _ptr(nq))
        self.n_qubits = nq

    def __del__(self):
        if getattr(self, "_h", None) is not None:
            lib().orc_program_free(self._h)
            self._h = None

    def _theta(self, theta):
        th = np.ascontiguousarray(np.asarray(theta, dtype=np.float64).reshape(self.B, self.S))
        if self.S == 0:
            th = np.zeros((self.B, 1), dtype=np.float64)
        return th


class Observables:
    def __init__(self, blob: bytes):
        h = ctypes.c_void_p()
        _check(lib().orc_obs_parse(blob, len(blob), ctypes.byref(h)))
        self._h = h
        import struct
        _, _, self.B, self.K = struct.unpack_from("<4sIII", blob, 0)

    def __del__(self):
        if getattr(self, "_h", None) is not None:
            lib().orc_obs_free(self._h)
            self._h = None


def simulate_state(prog: Program, theta):
    out = np.zeros((prog.B, 1 << prog.nmax), dtype=np.complex128)
    _check(lib().orc_simulate_state(prog._h, _ptr(prog._theta(theta)), _ptr(out)))
    return out


def expectation(prog: Program, theta, obs: Observables, return_imag=False):
    out = np.zeros((prog.B, obs.K), dtype=np.float64)
    im = np.zeros((prog.B, obs.K), dtype=np.float64)
    _check(lib().orc_expectation(prog._h, _ptr(prog._theta(theta)), obs._h, _ptr(out), _ptr(im)))
    return (out, im) if return_imag else out


def adjoint_grad(prog: Program, theta, obs: Observables, upstream):
    up = np.ascontiguousarray(np.asarray(upstream, dtype=np.float64).reshape(prog.B, obs.K))
    g = np.zeros((prog.B, max(prog.S, 1)), dtype=np.float64)
    _check(lib().orc_adjoint_grad(prog._h, _ptr(prog._theta(theta)), obs._h, _ptr(up), _ptr(g)))
    return g[:, : prog.S]


def amplitudes(prog: Program, theta, bitstrings):
    bs = np.ascontiguousarray(np.asarray(bitstrings, dtype=np.uint64).reshape(prog.B, -1))
    out = np.zeros(bs.shape, dtype=np.complex128)
    _check(lib().orc_amplitudes(prog._h, _ptr(prog._theta(theta)), _ptr(bs), bs.shape[1], _ptr(out)))
    return out


def sample(prog: Program, theta, n_shots, seed):
    out = np.zeros((prog.B, n_shots), dtype=np.uint64)
    _check(lib().orc_sample(prog._h, _ptr(prog._theta(theta)), n_shots, ctypes.c_uint64(seed), _ptr(out)))
    return out


def sample_from_state(states_c64, n_shots, seed):
    st = np.ascontiguousarray(np.asarray(states_c64, dtype=np.complex64))
    B, N = st.shape
    n = int(N).bit_length() - 1
    assert (1 << n) == N
    out = np.zeros((B, n_shots), dtype=np.uint64)
    _check(lib().orc_sample_from_state(_ptr(st), B, n, n_shots, ctypes.c_uint64(seed), _ptr(out)))
    return out


def gate_matrix(op, params=(), explicit=None):
    p = np.zeros(2, dtype=np.float64)
    p[: len(params)] = params
    ex = np.zeros(32, dtype=np.float64) if explicit is None else np.ascontiguousarray(
        np.stack([np.real(explicit).ravel(), np.imag(explicit).ravel()], axis=1).ravel(), dtype=np.float64)
    if ex.size < 32:
        ex = np.concatenate([ex, np.zeros(32 - ex.size)])
    out = np.zeros(32, dtype=np.float64)
    d = ctypes.c_int()
    _check(lib().orc_gate_matrix(op, _ptr(p), _ptr(ex), _ptr(out), ctypes.byref(d)))
    m = out[: 2 * d.value * d.value].view(np.complex128)
    return m.reshape(d.value, d.value).copy()


def gate_dmatrix(op, params, which=0):
    p = np.zeros(2, dtype=np.float64)
    p[: len(params)] = params
    out = np.zeros(32, dtype=np.float64)
    d = ctypes.c_int()
    _check(lib().orc_gate_dmatrix(op, _ptr(p), which, _ptr(out), ctypes.byref(d)))
    m = out[: 2 * d.value * d.value].view(np.complex128)
    return m.reshape(d.value, d.value).copy()


def splitmix64(seed, counter):
    return int(lib().orc_splitmix64(ctypes.c_uint64(seed), ctypes.c_uint64(counter)))


def set_c64_storage(on):
    lib().orc_set_c64_storage(1 if on else 0)


def num_threads():
    return int(lib().orc_num_threads())


def set_noise_seed(seed):
    """Seed of the channels' Kraus draws in every later call (trajectory rows)."""
    lib().orc_set_noise_seed(int(seed) & 0xFFFFFFFFFFFFFFFF)


def channel_pick(seed, row, chan, px, py, pz):
    """The Pauli (0 = I, 1 = X, 2 = Y, 3 = Z) channel `chan` of batch row `row` applies."""
    return int(lib().orc_channel_pick(int(seed) & 0xFFFFFFFFFFFFFFFF, int(row), int(chan), float(px), float(py),
                                      float(pz)))


def set_row_offset(offset):
    """Rows of a program draw their channels as rows offset + b of a larger batch."""
    lib().orc_set_row_offset(int(offset))


def sampled_expectation(prog: Program, theta, obs: Observables, reps, seed):
    """[B, K] expectations estimated from `reps` shots per non-identity term."""
    out = np.zeros((prog.B, obs.K), dtype=np.float64)
    _check(lib().orc_sampled_expectation(prog._h, _ptr(prog._theta(theta)), obs._h, int(reps),
                                         int(seed) & 0xFFFFFFFFFFFFFFFF, _ptr(out)))
    return out


def sampled_from_terms(obs: Observables, term_exp, reps, seed):
    """The same estimate from given float32 term expectations [B, Kt] (the
    j-th non-identity term of each row over (k, t) in order)."""
    te = np.ascontiguousarray(np.asarray(term_exp, dtype=np.float32))
    out = np.zeros((obs.B, obs.K), dtype=np.float64)
    _check(lib().orc_sampled_from_terms(obs._h, _ptr(te), te.shape[1], int(reps), int(seed) & 0xFFFFFFFFFFFFFFFF,
                                        _ptr(out)))
    return out


def param_shift_grad(prog: Program, theta, obs: Observables, upstream, reps=0, seed=0):
    """[B, S] gradients of sum_k g_k <h_k> by the parameter-shift rule, every
    symbolic parameter shifted alone; reps > 0 estimates each shifted
    circuit's expectations from that many shots per term."""
    up = np.ascontiguousarray(np.asarray(upstream, dtype=np.float64))
    g = np.zeros((prog.B, prog.S), dtype=np.float64)
    _check(lib().orc_param_shift_grad(prog._h, _ptr(prog._theta(theta)), obs._h, _ptr(up), int(reps),
                                      int(seed) & 0xFFFFFFFFFFFFFFFF, _ptr(g)))
    return g


def finite_diff_grad(prog: Program, theta, obs: Observables, upstream, eps):
    """[B, S] gradients by central differences of step eps in each symbol."""
    up = np.ascontiguousarray(np.asarray(upstream, dtype=np.float64))
    g = np.zeros((prog.B, prog.S), dtype=np.float64)
    _check(lib().orc_finite_diff_grad(prog._h, _ptr(prog._theta(theta)), obs._h, _ptr(up), float(eps), _ptr(g)))
    return g
