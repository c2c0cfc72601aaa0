"""tq_sample_from_state_noalloc (no allocation; static device workspace)
against tq_sample_from_state: bit-identical samples on two calls in a row,
the second with a smaller input, and the size limit rejected on the host."""
import numpy as np
import pytest
import torch

from gpu_util import dev, say
from paper_2003_02989_amd import tq

pytestmark = pytest.mark.gpu


def _states(rng, B, n):
    z = (rng.standard_normal((B, 1 << n)) + 1j * rng.standard_normal((B, 1 << n))).astype(np.complex64)
    z /= np.linalg.norm(z, axis=1, keepdims=True)
    z = z.astype(np.complex64)
    z[-1, ::5] = 0
    return dev(z, torch.complex64)


def test_noalloc_matches_allocating_sampler():
    rng = np.random.default_rng(42)
    # two calls in a row, the second smaller: the shared static workspace
    # keeps the first call's contents, which the second must not see
    for B, n, shots, seed in ((6, 20, 30000, 11), (3, 9, 5000, 12)):
        st = _states(rng, B, n)
        ref = tq.sample_from_state(st, shots, seed)
        out = torch.empty((B, shots), dtype=torch.int64, device="cuda")
        got = tq.sample_from_state_noalloc(st, shots, seed, out)
        torch.cuda.synchronize()
        say("noalloc B", B, "n", n, "mismatches", int((got != ref).sum().item()))
        assert torch.equal(got, ref)
    # the limit: B * (2^n / 64 + ...) level entries <= 2^22, checked before any launch
    big = torch.zeros((1, 1 << 28), dtype=torch.complex64, device="cuda")
    out = torch.empty((1, 4), dtype=torch.int64, device="cuda")
    with pytest.raises(tq.TQError) as e:
        tq.sample_from_state_noalloc(big, 4, 1, out)
    assert e.value.status == tq.TQ_E_UNSUPPORTED
