"""Write workload5_oracle.npz: the CPU oracle's peak and cost of every one of
the 4096 candidates of the random-DAG workload (n = 4001, seed 4), for the
GPU parity test that compares all of them.

Calls only the oracle (and the seeded input generator). Candidates are
independent, so they are split over worker processes; each runs the
unmodified oracle on its own candidates.

    python tests/golden/make_workload5_fixture.py [--workers N]
"""
import argparse
import os
import sys
import time
from multiprocessing import Pool

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import ref  # noqa: E402
from paper_1910_02653_amd import workloads as wl  # noqa: E402

OUT = os.path.join(HERE, "workload5_oracle.npz")

_w = None
_q = None


def _init():
    global _w, _q
    _w = wl.config(5)
    _q = ref.quantize(_w.s_frac)


def _one(k):
    return ref.eval_candidate(_w, k, q=_q)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workers", type=int, default=os.cpu_count() or 1)
    args = ap.parse_args()
    w = wl.config(5)
    t0 = time.time()
    with Pool(args.workers, initializer=_init) as pool:
        res = pool.map(_one, range(w.K), chunksize=8)
    peak = np.array([r[0] for r in res], np.int64)
    cost = np.array([r[1] for r in res], np.int64)
    np.savez_compressed(OUT, peak=peak, cost=cost, n=np.int64(w.n), K=np.int64(w.K), seed=np.int64(w.seed))
    print("wrote %s: %d candidates in %.0f s" % (OUT, w.K, time.time() - t0))


if __name__ == "__main__":
    main()
