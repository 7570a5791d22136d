"""Find the expert-0 logit bias of the prefill-scale skewed workload.

The workload (T=16384, d=4096, E=16) asks that expert 0 receive about 40% of
the tokens while experts 1..15 follow a Zipf(1.2) prior.  The bias of
experts 1..15 is fixed (-1.2 ln e); this script bisects the expert-0 bias on
the oracle's own router logits at seed 0 and prints the value stored as
``SKEW_BIAS0`` in paper_2410_19123_amd/workloads.py.  It calls only the
oracle and the input generator.

    python -m oracle.calibrate_skew_bias
"""
import numpy as np

from oracle import oracle
from paper_2410_19123_amd import workloads as wl


def main(target: float = 0.40, seed: int = 0):
    w = wl.WORKLOADS["prefill_skew16"]
    x = wl.make_x(w, seed)
    wr, b = wl.make_router(w, seed)
    b = b.copy()
    b[0] = 0.0
    _, logits = oracle.route(x, wr, b)
    s0 = logits[:, 0].astype(np.float64)
    rest = logits[:, 1:].max(axis=1).astype(np.float64)
    lo, hi = -10.0, 10.0
    for _ in range(80):
        mid = 0.5 * (lo + hi)
        frac = np.mean(s0 + mid >= rest)
        lo, hi = (lo, mid) if frac > target else (mid, hi)
    v = round(0.5 * (lo + hi), 4)
    b[0] = v
    ids, _ = oracle.route(x, wr, b)
    counts = np.bincount(ids, minlength=w.E)
    print(f"SKEW_BIAS0 = {v}")
    print("share of expert 0:", counts[0] / w.T)
    print("counts:", counts.tolist())
    return v


if __name__ == "__main__":
    main()
