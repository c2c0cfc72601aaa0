"""Write tests/golden/c4_n30.npz from the oracle (CPU, complex128).

The 30-qubit random circuit (5x6 grid, depth 20, seed 200302989 + 4) is too
large to simulate inside a test, so this script runs the oracle once and
stores: the 4096 amplitudes at the workload's seeded bitstrings, the squared
norm, and sum_i p_i^2 (the mean of 2^n p(x) over exact samples is
2^n sum_i p_i^2).  It calls only oracle/ and the input generators.

    OMP_NUM_THREADS=8 python tests/golden/make_c4_golden.py
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as orc  # noqa: E402
from paper_2003_02989_amd import workloads as wl  # noqa: E402


def main(out=os.path.join(ROOT, "tests", "golden", "c4_n30.npz")):
    orc.build()
    w = wl.c4_random()
    prog = orc.Program(w.program_blob())
    t0 = time.time()
    st = orc.simulate_state(prog, np.zeros((1, 0)))[0]
    t1 = time.time()
    bits = w.extras["bitstrings"][0]
    amps = st[bits.astype(np.int64)]
    norm2 = 0.0
    sum_p2 = 0.0
    chunk = 1 << 24
    for i in range(0, st.size, chunk):
        p = np.abs(st[i:i + chunk]) ** 2
        norm2 += float(p.sum())
        sum_p2 += float((p * p).sum())
    np.savez(out, bitstrings=bits, amplitudes=amps, norm2=norm2, sum_p2=sum_p2, n=30,
             oracle_seconds=t1 - t0, threads=orc.num_threads())
    print(f"wrote {out}: oracle {t1 - t0:.1f} s on {orc.num_threads()} threads, norm2 {norm2:.15f}, "
          f"2^n sum p^2 {sum_p2 * 2.0 ** 30:.6f}")


if __name__ == "__main__":
    main()
