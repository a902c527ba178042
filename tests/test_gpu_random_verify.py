"""GPU parity of sense_soft_gate_verify over seeded random shapes and gate
parameters: vocabulary (1 to 200K, multiples of the vector width or not),
draft length 1-64, candidates and groups, logits type, ragged draft lengths
(clamped at both ends) with out-of-vocabulary ids, and gamma, top-k, window,
tolerance and entropy normalisation drawn from their ranges.  Every case
meets the oracle under the rules of tests/parity.py (ranks and the em /
top-k / window bits exactly, gate scores within GATE_ABS, accepted lengths
and best drafts exactly away from gamma).  Shapes come from a fixed seed and
are printed before each case."""
import numpy as np
import pytest
import torch

from test_gpu_verify import run, structured

pytestmark = pytest.mark.gpu

VOCABS = [1, 2, 7, 64, 77, 1000, 1001, 4099, 32000, 65537, 128256, 152064, 200003]


def shapes(count=64, seed=20261203):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        v = int(rng.choice(VOCABS))
        m = int(rng.choice([1, 2, 5, 8, 12, 31, 64]))
        groups = int(rng.choice([1, 2, 3, 4]))
        c = groups * int(rng.integers(1, 12))
        if c * m * v > 6e7:                          # keep the oracle's pass over the logits short
            continue
        dtype = str(rng.choice(["f32", "f16", "bf16"]))
        gamma = float(rng.choice([0.0, 0.01, 0.05, 0.2, 0.9, 1.5]))
        topk = int(rng.choice([1, 2, 3, 10, 1 << 20]))
        window = int(rng.integers(0, min(m, 64) + 1))
        tau = int(rng.integers(0, 3))
        normed = bool(rng.random() < 0.8)
        ragged = bool(rng.random() < 0.5)
        out.append((c, m, v, groups, dtype, gamma, topk, window, tau, normed, ragged))
    return out


CASES = shapes()


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_random_verify_matches_oracle(case):
    c, m, v, groups, dtype, gamma, topk, window, tau, normed, ragged = case
    print(f"[random-verify] C={c} M={m} V={v} groups={groups} {dtype} gamma={gamma} "
          f"topk={topk} W={window} tau={tau} normalised={normed} ragged={ragged}", flush=True)
    seed = (c * 31 + m * 7 + v) % 100003
    logits, drafts = structured(seed, c, m, v, p_match=0.8, dtype=dtype)
    lens = None
    if ragged:
        rng = np.random.default_rng(seed)
        lens = rng.integers(-1, m + 2, c).astype(np.int32)   # clamped to [0, m]
        bad = rng.random((c, m)) < 0.05
        drafts = torch.where(torch.from_numpy(bad), torch.full_like(drafts, v), drafts)
    run(logits, drafts, lens, n_groups=groups, gamma=gamma, topk=topk, window=window, tau=tau,
        entropy_normalized=normed)
