"""Python binding of libtq: argument marshalling only.

Every function takes torch tensors that live on the current HIP device,
checks their dtype, shape and contiguity, and passes raw device pointers and
the current stream to the C ABI declared in include/tq.h.  All arithmetic
happens in the library's HIP kernels; there is no fallback: if libtq.so
cannot be loaded every call raises.
"""
import ctypes
import os
import struct

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# TQ_LIB_PATH: another build of the same sources (the sanitizer test loads one)
LIB_PATH = os.environ.get("TQ_LIB_PATH") or os.path.join(_HERE, "libtq.so")

TQ_OK, TQ_E_INVALID, TQ_E_UNSUPPORTED, TQ_E_NOMEM, TQ_E_DEVICE = range(5)
_STATUS = {1: "TQ_E_INVALID", 2: "TQ_E_UNSUPPORTED", 3: "TQ_E_NOMEM", 4: "TQ_E_DEVICE"}


class TQError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class _Options(ctypes.Structure):
    _fields_ = [("max_tile_qubits", ctypes.c_int32), ("low_qubits", ctypes.c_int32),
                ("fuse", ctypes.c_int32), ("max_pass_gates", ctypes.c_int32), ("specialize", ctypes.c_int32)]


_lib = None


def lib():
    """Load libtq.so (raises OSError when it is missing: there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OSError(f"{LIB_PATH} is missing: build it with `python -m paper_2003_02989_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
        p32 = ctypes.POINTER(ctypes.c_int32)
        L.tq_last_error.restype = ctypes.c_char_p
        L.tq_version.restype = ctypes.c_char_p
        L.tq_program_create.argtypes = [ctypes.c_char_p, sz, ctypes.POINTER(_Options), ctypes.POINTER(vp)]
        L.tq_program_destroy.argtypes = [vp]
        L.tq_program_destroy.restype = None
        L.tq_program_info.argtypes = [vp, p32, p32, p32, p32]
        L.tq_program_specialize.argtypes = [vp, ctypes.c_char_p]
        L.tq_program_set_noise_seed.argtypes = [vp, u64]
        L.tq_row_mean.argtypes = [vp, i64, i32, i32, vp, vp]
        L.tq_observables_create.argtypes = [ctypes.c_char_p, sz, ctypes.POINTER(vp)]
        L.tq_observables_destroy.argtypes = [vp]
        L.tq_observables_destroy.restype = None
        L.tq_observables_info.argtypes = [vp, p32, p32]
        L.tq_simulate_state.argtypes = [vp, vp, vp, vp]
        L.tq_expectation.argtypes = [vp, vp, vp, vp, vp]
        L.tq_sample.argtypes = [vp, vp, i64, u64, vp, vp]
        L.tq_sample_with_amplitudes.argtypes = [vp, vp, i64, u64, vp, vp, i64, vp, vp]
        L.tq_adjoint_grad.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.tq_amplitudes.argtypes = [vp, vp, vp, i64, vp, vp]
        L.tq_sample_from_state.argtypes = [vp, i32, i32, i64, u64, vp, vp]
        L.tq_sample_from_state_noalloc.argtypes = [vp, i32, i32, i64, u64, vp, vp]
        L.tq_amplitudes_from_state.argtypes = [vp, i32, i32, vp, i64, vp, vp]
        L.tq_program_describe.argtypes = [vp, ctypes.c_char_p, sz, ctypes.POINTER(sz)]
        L.tq_build_matrices.argtypes = [vp, vp, vp, i64, ctypes.POINTER(i64), vp]
        L.tq_gate_matrix.argtypes = [i32, vp, vp, i32, i32, i32, vp, p32, ctypes.POINTER(ctypes.c_double)]
        L.tq_observables_terms.argtypes = [vp, p32]
        L.tq_sampled_expectation.argtypes = [vp, vp, vp, i32, u64, vp, vp, vp]
        L.tq_param_shift_grad.argtypes = [vp, vp, vp, vp, i32, u64, vp, vp]
        L.tq_finite_diff_grad.argtypes = [vp, vp, vp, vp, ctypes.c_double, vp, vp]
        L.tq_profile_start.argtypes = [ctypes.c_char_p]
        L.tq_profile_read.argtypes = [ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_double)]
        for f in ("tq_program_create", "tq_program_info", "tq_program_specialize", "tq_observables_create", "tq_observables_info",
                  "tq_simulate_state", "tq_expectation", "tq_sample", "tq_sample_with_amplitudes", "tq_adjoint_grad",
                  "tq_amplitudes",
                  "tq_sample_from_state", "tq_sample_from_state_noalloc", "tq_amplitudes_from_state", "tq_program_describe", "tq_profile_start", "tq_profile_read",
                  "tq_gate_matrix", "tq_build_matrices", "tq_observables_terms", "tq_sampled_expectation",
                  "tq_param_shift_grad", "tq_finite_diff_grad"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc):
    if rc != TQ_OK:
        raise TQError(rc, lib().tq_last_error().decode())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, dtype, shape, name):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


class Program:
    """A parsed and planned batch of circuits (``tq_program``)."""

    def __init__(self, blob: bytes, max_tile_qubits=0, low_qubits=0, fuse=True, max_pass_gates=0, specialize=False):
        opt = _Options(max_tile_qubits, low_qubits, 1 if fuse else -1, max_pass_gates, 1 if specialize else 0)
        h = ctypes.c_void_p()
        _check(lib().tq_program_create(blob, len(blob), ctypes.byref(opt), ctypes.byref(h)))
        self._h = h
        B, S, n = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib().tq_program_info(h, ctypes.byref(B), ctypes.byref(S), ctypes.byref(n), None))
        self.B, self.S, self.max_qubits = B.value, S.value, n.value
        q = (ctypes.c_int32 * max(self.B, 1))()
        _check(lib().tq_program_info(h, None, None, None, q))
        self.qubits = list(q)[: self.B]

    def close(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.tq_program_destroy(h)

    __del__ = close


class Observables:
    """B x K Pauli sums (``tq_observables``)."""

    def __init__(self, blob: bytes):
        h = ctypes.c_void_p()
        _check(lib().tq_observables_create(blob, len(blob), ctypes.byref(h)))
        self._h = h
        self.B, self.K = struct.unpack_from("<II", blob, 8)

    def close(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.tq_observables_destroy(h)

    __del__ = close


def specialize(prog, target=None):
    """Compile the program's structure-specialised kernels now (for the
    current device, or only check them for an offload target such as
    "gfx950" when `target` is given)."""
    _check(lib().tq_program_specialize(prog._h, target.encode() if target else None))


def describe(prog):
    """The plan of a program as a dict (tq_program_describe)."""
    import json
    need = ctypes.c_size_t()
    _check(lib().tq_program_describe(prog._h, None, 0, ctypes.byref(need)))
    buf = ctypes.create_string_buffer(need.value)
    _check(lib().tq_program_describe(prog._h, buf, need.value, None))
    return json.loads(buf.value.decode())


def build_matrices(prog, symbol_values, stream=None):
    """The device builder's matrix blocks (tq_build_matrices): complex128
    device tensor of every group's rows x mat_block entries, concatenated."""
    need = ctypes.c_int64()
    _check(lib().tq_build_matrices(prog._h, None, None, 0, ctypes.byref(need), None))
    out = torch.empty(max(need.value, 1), dtype=torch.complex128, device="cuda")
    _check(lib().tq_build_matrices(prog._h, _theta(prog, symbol_values), ctypes.c_void_p(out.data_ptr()), need.value,
                                   None, _stream(stream)))
    return out[: need.value]


def gate_matrix(op, params=(), explicit=None, cblock=False, deriv=False, which=0):
    """(matrix, phase) of the library's gate table (tq_gate_matrix, host
    only): numpy complex128 [d, d] as the builder forms it and the global
    phase it leaves out (the gate's matrix is exp(1j * phase) * matrix)."""
    import numpy as np
    p = np.zeros(2, dtype=np.float64)
    p[: len(params)] = params
    ex = None
    if explicit is not None:
        m = np.asarray(explicit, np.complex128).ravel()
        ex = np.ascontiguousarray(np.stack([m.real, m.imag], axis=1).ravel())
    out = np.zeros(32, dtype=np.float64)
    d = ctypes.c_int32()
    ph = ctypes.c_double()
    _check(lib().tq_gate_matrix(int(op), ctypes.c_void_p(p.ctypes.data),
                                ctypes.c_void_p(ex.ctypes.data) if ex is not None else None, 1 if cblock else 0,
                                1 if deriv else 0, int(which), ctypes.c_void_p(out.ctypes.data), ctypes.byref(d),
                                ctypes.byref(ph)))
    k = d.value
    return out[: 2 * k * k].view(np.complex128).reshape(k, k).copy(), ph.value


def profile_start(kernel):
    _check(lib().tq_profile_start(kernel.encode() if kernel else None))


def profile_read():
    """(launches, total_ms) of the bracketed launches since profile_start."""
    n, ms = ctypes.c_int64(), ctypes.c_double()
    _check(lib().tq_profile_read(ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value


def _theta(prog, symbol_values):
    if prog.S == 0:
        return None
    return _dev(symbol_values, torch.float32, (prog.B, prog.S), "symbol_values")


def simulate_state(prog, symbol_values, out=None, stream=None):
    if out is None:
        out = torch.empty((prog.B, 1 << prog.max_qubits), dtype=torch.complex64, device="cuda")
    p = _dev(out, torch.complex64, (prog.B, 1 << prog.max_qubits), "states")
    _check(lib().tq_simulate_state(prog._h, _theta(prog, symbol_values), p, _stream(stream)))
    return out


def set_noise_seed(prog, seed):
    """Seed of the channels' per-row Kraus draws in the program's later calls."""
    _check(lib().tq_program_set_noise_seed(prog._h, int(seed) & 0xFFFFFFFFFFFFFFFF))


def row_mean(x, R, out=None, stream=None):
    """[G R, K] float32 -> [G, K]: the mean over each R consecutive rows (the
    trajectories of one noisy circuit)."""
    G = x.shape[0] // R
    if x.shape[0] != G * R:
        raise ValueError("rows must be a multiple of R")
    K = x.shape[1]
    if out is None:
        out = torch.empty((G, K), dtype=torch.float32, device="cuda")
    i = _dev(x, torch.float32, (G * R, K), "in")
    o = _dev(out, torch.float32, (G, K), "out")
    _check(lib().tq_row_mean(i, G, R, K, o, _stream(stream)))
    return out


def expectation(prog, symbol_values, obs, out=None, stream=None):
    if out is None:
        out = torch.empty((prog.B, obs.K), dtype=torch.float32, device="cuda")
    p = _dev(out, torch.float32, (prog.B, obs.K), "out")
    _check(lib().tq_expectation(prog._h, _theta(prog, symbol_values), obs._h, p, _stream(stream)))
    return out


def adjoint_grad(prog, symbol_values, obs, upstream, grad=None, expectations=None, stream=None):
    """Returns grad [B, S]; fills `expectations` [B, K] too when given."""
    if grad is None:
        grad = torch.empty((prog.B, prog.S), dtype=torch.float32, device="cuda")
    g = _dev(grad, torch.float32, (prog.B, prog.S), "grad") if prog.S else None
    u = _dev(upstream, torch.float32, (prog.B, obs.K), "upstream")
    e = _dev(expectations, torch.float32, (prog.B, obs.K), "expectations")
    _check(lib().tq_adjoint_grad(prog._h, _theta(prog, symbol_values), obs._h, u, g, e, _stream(stream)))
    return grad


def observables_terms(obs):
    """Kt: the most non-identity terms any row of `obs` has."""
    kt = ctypes.c_int32()
    _check(lib().tq_observables_terms(obs._h, ctypes.byref(kt)))
    return kt.value


def sampled_expectation(prog, symbol_values, obs, reps, seed, out=None, term_out=None, stream=None):
    """[B, K] expectations estimated from `reps` shots per non-identity term
    (tq_sampled_expectation); `term_out` [B, Kt] receives the term values the
    shots were drawn from when given."""
    if out is None:
        out = torch.empty((prog.B, obs.K), dtype=torch.float32, device="cuda")
    p = _dev(out, torch.float32, (prog.B, obs.K), "out")
    t = _dev(term_out, torch.float32, (prog.B, observables_terms(obs)), "term_out") if term_out is not None else None
    _check(lib().tq_sampled_expectation(prog._h, _theta(prog, symbol_values), obs._h, int(reps),
                                        ctypes.c_uint64(int(seed) & 0xFFFFFFFFFFFFFFFF), p, t, _stream(stream)))
    return out


def param_shift_grad(prog, symbol_values, obs, upstream, reps=0, seed=0, grad=None, stream=None):
    """[B, S] gradients by the parameter-shift rule (tq_param_shift_grad);
    reps > 0 takes each shifted circuit's expectations from that many shots
    per term."""
    if grad is None:
        grad = torch.empty((prog.B, prog.S), dtype=torch.float32, device="cuda")
    g = _dev(grad, torch.float32, (prog.B, prog.S), "grad") if prog.S else None
    u = _dev(upstream, torch.float32, (prog.B, obs.K), "upstream")
    _check(lib().tq_param_shift_grad(prog._h, _theta(prog, symbol_values), obs._h, u, int(reps),
                                     ctypes.c_uint64(int(seed) & 0xFFFFFFFFFFFFFFFF), g, _stream(stream)))
    return grad


def finite_diff_grad(prog, symbol_values, obs, upstream, eps, grad=None, stream=None):
    """[B, S] gradients by central differences of step eps (tq_finite_diff_grad)."""
    if grad is None:
        grad = torch.empty((prog.B, prog.S), dtype=torch.float32, device="cuda")
    g = _dev(grad, torch.float32, (prog.B, prog.S), "grad") if prog.S else None
    u = _dev(upstream, torch.float32, (prog.B, obs.K), "upstream")
    _check(lib().tq_finite_diff_grad(prog._h, _theta(prog, symbol_values), obs._h, u, float(eps), g,
                                     _stream(stream)))
    return grad


def sample(prog, symbol_values, n_shots, seed, out=None, stream=None):
    """Bitstrings as int64 [B, n_shots] (the bit patterns of the uint64 output)."""
    if out is None:
        out = torch.empty((prog.B, n_shots), dtype=torch.int64, device="cuda")
    p = _dev(out, torch.int64, (prog.B, n_shots), "out")
    _check(lib().tq_sample(prog._h, _theta(prog, symbol_values), int(n_shots), ctypes.c_uint64(seed), p,
                           _stream(stream)))
    return out


def amplitudes(prog, symbol_values, bitstrings, out=None, stream=None):
    M = bitstrings.shape[1]
    b = _dev(bitstrings, torch.int64, (prog.B, M), "bitstrings")
    if out is None:
        out = torch.empty((prog.B, M), dtype=torch.complex64, device="cuda")
    p = _dev(out, torch.complex64, (prog.B, M), "amps")
    _check(lib().tq_amplitudes(prog._h, _theta(prog, symbol_values), b, M, p, _stream(stream)))
    return out


def sample_with_amplitudes(prog, symbol_values, n_shots, seed, bitstrings, out=None, amps=None, stream=None):
    """One simulation, both outputs: (samples int64 [B, n_shots], amplitudes
    complex64 [B, M]) at bitstrings int64 [B, M]."""
    M = bitstrings.shape[1]
    b = _dev(bitstrings, torch.int64, (prog.B, M), "bitstrings")
    if out is None:
        out = torch.empty((prog.B, n_shots), dtype=torch.int64, device="cuda")
    if amps is None:
        amps = torch.empty((prog.B, M), dtype=torch.complex64, device="cuda")
    p = _dev(out, torch.int64, (prog.B, n_shots), "out")
    a = _dev(amps, torch.complex64, (prog.B, M), "amps")
    _check(lib().tq_sample_with_amplitudes(prog._h, _theta(prog, symbol_values), int(n_shots), ctypes.c_uint64(seed),
                                           p, b, M, a, _stream(stream)))
    return out, amps


def sample_from_state(states, n_shots, seed, out=None, stream=None):
    B, N = states.shape
    n = N.bit_length() - 1
    if (1 << n) != N:
        raise ValueError("state length must be a power of two")
    s = _dev(states, torch.complex64, (B, N), "states")
    if out is None:
        out = torch.empty((B, n_shots), dtype=torch.int64, device="cuda")
    p = _dev(out, torch.int64, (B, n_shots), "out")
    _check(lib().tq_sample_from_state(s, B, n, int(n_shots), ctypes.c_uint64(seed), p, _stream(stream)))
    return out


def sample_from_state_noalloc(states, n_shots, seed, out, stream=None):
    """sample_from_state without any allocation (tq_sample_from_state_noalloc):
    `out` int64 [B, n_shots] is required."""
    B, N = states.shape
    n = N.bit_length() - 1
    if (1 << n) != N:
        raise ValueError("state length must be a power of two")
    s = _dev(states, torch.complex64, (B, N), "states")
    p = _dev(out, torch.int64, (B, n_shots), "out")
    _check(lib().tq_sample_from_state_noalloc(s, B, n, int(n_shots), ctypes.c_uint64(seed), p, _stream(stream)))
    return out


def amplitudes_from_state(states, bitstrings, out=None, stream=None):
    """Amplitudes [B, M] of given states [B, 2^n] at bitstrings int64 [B, M]."""
    B, N = states.shape
    n = N.bit_length() - 1
    if (1 << n) != N:
        raise ValueError("state length must be a power of two")
    M = bitstrings.shape[1]
    s = _dev(states, torch.complex64, (B, N), "states")
    b = _dev(bitstrings, torch.int64, (B, M), "bitstrings")
    if out is None:
        out = torch.empty((B, M), dtype=torch.complex64, device="cuda")
    p = _dev(out, torch.complex64, (B, M), "amps")
    _check(lib().tq_amplitudes_from_state(s, B, n, b, M, p, _stream(stream)))
    return out
