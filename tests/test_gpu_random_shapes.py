"""GPU parity of sense_retrieve over seeded random shapes, so that no
dispatch boundary is only ever met at the sizes picked by hand: key dimension
(multiples of 8 from 8 to 4096, short and long keys), store size (both sides
of the direct / sampled-threshold boundary of batches, ragged selection
chunks), batch size (one query, two and three, partial and whole 16-query
tiles, two query groups), k (1 to 1024), metric, key type, ragged
continuations and padded row strides.  Every case meets the oracle under the
rules of tests/parity.py (ordered ids up to bounded near ties, scores within
their derived bounds, drafts exactly).  The shapes come from a fixed seed and
are printed before each case."""
import numpy as np
import pytest

from paper_2606_00021_amd import synth
from test_gpu_retrieval import run_case

pytestmark = pytest.mark.gpu

DIMS = [8, 16, 24, 40, 56, 64, 72, 128, 200, 256, 520, 1000, 1024, 2056, 4096]
BATCHES = [1, 1, 1, 2, 3, 5, 16, 17, 33, 64, 65]


def shapes(count=64, seed=20261202):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        d = int(rng.choice(DIMS))
        nq = int(rng.choice(BATCHES))
        if rng.random() < 0.3 and d <= 256:
            n = int(rng.integers(131_073, 200_000))     # sampled threshold for batches
        else:
            n = int(rng.integers(1, 60_000))
        # keep the oracle's fp64 scan of every row to about a second, and
        # enough rows for a batch's queries to come from distinct clusters
        if n * d * nq > 1.2e9 or (nq > 1 and n < 8 * max(64, 2 * nq)):
            continue
        kmax = min(n, 1024)
        k = int(min(kmax, max(1, rng.choice([1, 8, 64, 100, 128, 512, 1024]))))
        metric = "cosine" if rng.random() < 0.6 else "ip"
        kdt = "bf16" if rng.random() < 0.5 else "f16"
        stride = d + 8 * int(rng.integers(1, 4)) if rng.random() < 0.2 else None
        ragged = bool(rng.random() < 0.4)
        out.append((n, d, kdt, nq, k, metric, stride, ragged))
    return out


CASES = shapes()


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_random_shape_matches_oracle(case):
    n, d, kdt, nq, k, metric, stride, ragged = case
    print(f"[random-shape] n={n} d={d} {kdt} nq={nq} k={k} {metric} stride={stride} "
          f"ragged={ragged}", flush=True)
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], name=f"random-{n}-{d}-{nq}", n=n, d=d,
                     key_dtype=kdt, k=k, n_queries=nq, n_clusters=max(64, 2 * nq),
                     n_outliers=min(4, d // 8))
    run_case(w, seed=n % 9973 + d, metric=metric, key_stride=stride, ragged_spans=ragged)
