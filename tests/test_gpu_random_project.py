"""GPU parity of sense_project over seeded random shapes: rows (the direct
route below 256 rows, the matrix-core route above), input dimension
(multiples of 8 up to 4096, ragged against the 32-dimension steps), output
dimension (1 to 256: the fused epilogue up to 64, the intermediate beyond),
input and output types, a mean or none, normalised or raw, and output rows
wider than d_out (one output per store or four).  Each case meets the oracle
within the bound of tests/test_gpu_project.py and leaves the columns past
d_out untouched.  Shapes come from a fixed seed and are printed first."""
import numpy as np
import pytest
import torch

from paper_2606_00021_amd import sense, synth
from parity import host_bits
from test_gpu_project import check_projection

pytestmark = pytest.mark.gpu
DEV = "cuda"


def shapes(count=32, seed=20261204):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        n = int(rng.choice([1, 7, 255, 256, 300, 1000, 2049, 5000]))
        d_in = 8 * int(rng.integers(1, 513))
        d_out = int(rng.choice([1, 3, 4, 8, 30, 40, 63, 64, 65, 100, 128, 256]))
        if d_out > d_in or n * d_in * d_out > 1e9:
            continue
        xdt = str(rng.choice(["bf16", "f16", "f32"]))
        odt = str(rng.choice(["bf16", "f16", "f32"]))
        with_mean = bool(rng.random() < 0.7)
        normalize = bool(rng.random() < 0.7)
        extra = int(rng.choice([0, 0, 1, 2, 4]))
        out.append((n, d_in, d_out, xdt, odt, with_mean, normalize, extra))
    return out


CASES = shapes()
TDT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_random_projection_matches_oracle(case):
    n, d_in, d_out, xdt, odt, with_mean, normalize, extra = case
    print(f"[random-project] n={n} d_in={d_in} d_out={d_out} x={xdt} out={odt} mean={with_mean} "
          f"normalize={normalize} extra={extra}", flush=True)
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=max(n, 64), d=d_in,
                     key_dtype=xdt if xdt != "f32" else "bf16", n_clusters=16,
                     n_outliers=min(4, d_in // 8))
    ds = synth.make_datastore(w, n + d_in, DEV)
    mean, basis = synth.make_pca_basis(ds, n + d_in, d_out, sample=min(4096, w.n))
    x = ds.keys[:n]
    if xdt == "f32":
        x = x.float().contiguous()
    out = torch.full((n, d_out + extra), 3.0, dtype=TDT[odt], device=DEV)
    sense.sense_project(x, basis, mean if with_mean else None, normalize, out=out[:, :d_out])
    torch.cuda.synchronize()
    check_projection(out[:, :d_out], host_bits(x), xdt, basis, mean if with_mean else None,
                     normalize, odt)
    if extra:
        assert (out[:, d_out:] == 3.0).all(), "columns past d_out were written"
