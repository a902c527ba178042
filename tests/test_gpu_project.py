"""GPU parity of the PCA projection (Alg. 2's k = L2Norm(PCA(h)); the
datastore projection of Sec. 3.2 Eq. 6 with the implementation details'
4096 -> 64 PCA) and of the short-key scan that searches the projected keys.

Projection: every output element within one unit in the last place of the
output type of the oracle's exact value, plus an fp32 accumulation bound
2^-14 * sum_t (|x_t| + |mean_t|) |w_ot| (divided by the row norm when
normalised).  Scans of projected keys follow the retrieval rules.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_00021_amd import sense, synth
from parity import check_topk, dt_name, host_bits

pytestmark = pytest.mark.gpu

DEV = "cuda"


def ulp(v, dt):
    """Unit in the last place of |v| in the output type."""
    a = np.abs(v)
    mant = {"f32": 23, "f16": 10, "bf16": 7}[dt]
    emin = {"f32": -126, "f16": -14, "bf16": -126}[dt]
    e = np.floor(np.log2(np.maximum(a, 2.0 ** emin)))
    return 2.0 ** (e - mant)


def check_projection(gpu, x_bits, x_dt, basis, mean, normalize, out_dt, x_stride=None, d_in=None):
    b = basis.cpu().numpy().astype(np.float64)
    mu = None if mean is None else mean.cpu().numpy().astype(np.float64)
    exact = oracle.project(x_bits, x_dt, b, mu, normalize, x_stride=x_stride, d_in=d_in)
    raw = oracle.project(x_bits, x_dt, b, mu, False, x_stride=x_stride, d_in=d_in)
    xs = oracle.decode(x_bits, x_dt) if x_dt != "f32" else x_bits.astype(np.float64)
    d = b.shape[1]
    xs = xs.reshape(-1, xs.shape[-1] if x_stride is None else x_stride)[:, :d]
    absx = np.abs(xs) + (0 if mu is None else np.abs(mu))
    bound = 2.0 ** -14 * (absx @ np.abs(b).T)
    if normalize:
        nrm = np.linalg.norm(raw, axis=1, keepdims=True)
        bound = bound / np.where(nrm > 0, nrm, 1.0)
    g = gpu.float().cpu().numpy().astype(np.float64)
    err = np.abs(g - exact)
    tol = ulp(exact, out_dt) + bound
    worst = np.unravel_index(np.argmax(err - tol), err.shape)
    assert (err <= tol).all(), f"projection error {err[worst]} > {tol[worst]} at {worst}"


PROJ_CASES = [
    # n, d_in, d_out, x dtype, out dtype, mean, normalize
    (4096, 4096, 64, "bf16", "bf16", True, True),     # matrix-core route, fused epilogue
    (3000, 1024, 64, "f16", "f16", True, True),
    (2001, 2048, 30, "bf16", "bf16", True, True),     # fused, one output per store
    (1500, 1000, 64, "f16", "f32", False, True),      # fused, fp32 16-byte stores, ragged d
    (999, 1024, 4, "bf16", "bf16", True, False),      # fused, one 4-output store per row
    (700, 4096, 100, "bf16", "f32", False, False),    # two query groups on the matrix cores
    (2500, 512, 256, "bf16", "f32", True, True),
    (7, 4096, 64, "bf16", "f32", True, True),         # direct route (few rows)
    (33, 2048, 64, "f32", "bf16", True, True),        # fp32 rows: direct route
    (300, 8192, 8, "f16", "f32", False, True),
]


@pytest.mark.parametrize("case", PROJ_CASES, ids=[str(i) for i in range(len(PROJ_CASES))])
def test_project_matches_oracle(case):
    n, d_in, d_out, xdt, odt, with_mean, normalize = case
    print(f"[project] case={case}", flush=True)
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=max(n, 64), d=d_in,
                     key_dtype=xdt if xdt != "f32" else "bf16", n_clusters=32)
    ds = synth.make_datastore(w, 41, DEV)
    mean, basis = synth.make_pca_basis(ds, 41, d_out)
    x = ds.keys[:n]
    if xdt == "f32":
        x = x.float().contiguous()
    out = sense.sense_project(x, basis, mean if with_mean else None, normalize,
                              out_dtype=synth.DTYPES[odt])
    torch.cuda.synchronize()
    check_projection(out, host_bits(x), xdt, basis, mean if with_mean else None, normalize, odt)


def test_project_strided_rows_and_output_stride():
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=600, d=1000, n_clusters=8)
    ds = synth.make_datastore(w, 5, DEV, key_stride=1012)     # stride % 8 != 0 -> direct route
    mean, basis = synth.make_pca_basis(ds, 5, 48)
    out = torch.full((600, 64), 5.0, dtype=torch.float32, device=DEV)
    sense.sense_project(ds.keys, basis, mean, True, out=out)
    torch.cuda.synchronize()
    store = ds.keys.as_strided((600, 1012), (1012, 1))
    check_projection(out[:, :48], host_bits(store), "f16", basis, mean, True, "f32",
                     x_stride=1012, d_in=1000)
    assert (out[:, 48:] == 5.0).all()


@pytest.mark.parametrize("cols", [42, 44])
def test_project_matrix_core_output_stride(cols):
    """The matrix-core route (16-byte aligned rows, row stride a multiple of
    8) into a wider output: 40 outputs per row at a stride of 42 (one
    output per store) or 44 (four per store); the columns past 40 keep
    their values."""
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=2000, d=1024, key_dtype="bf16",
                     n_clusters=8)
    ds = synth.make_datastore(w, 7, DEV)
    mean, basis = synth.make_pca_basis(ds, 7, 40)
    out = torch.full((2000, cols), 5.0, dtype=torch.bfloat16, device=DEV)
    sense.sense_project(ds.keys, basis, mean, True, out=out[:, :40])
    torch.cuda.synchronize()
    check_projection(out[:, :40], host_bits(ds.keys), "bf16", basis, mean, True, "bf16")
    assert (out[:, 40:] == 5.0).all()


def test_project_routes_agree():
    """The matrix-core route (many aligned rows) and the direct route (the
    same rows one block each, via an fp32 copy) both meet the oracle."""
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=1024, d=4096, key_dtype="bf16",
                     n_clusters=16)
    ds = synth.make_datastore(w, 6, DEV)
    mean, basis = synth.make_pca_basis(ds, 6, 64)
    a = sense.sense_project(ds.keys, basis, mean, True)
    b = sense.sense_project(ds.keys.float(), basis, mean, True)
    torch.cuda.synchronize()
    assert (a - b).abs().max().item() < 1e-3


SMALL_SCAN = [
    # n, d, key dtype, n_queries, k, metric
    (10007, 64, "bf16", 1, 16, "cosine"),
    (20000, 64, "f16", 3, 64, "ip"),
    (5000, 8, "bf16", 1, 8, "cosine"),
    (5001, 16, "f16", 2, 32, "cosine"),
    (4099, 24, "bf16", 1, 10, "ip"),
    (70001, 40, "bf16", 1, 64, "cosine"),
    (3000, 56, "f16", 1, 5, "cosine"),
    (9000, 64, "bf16", 16, 64, "cosine"),       # query batch: matrix-core scan at d = 64
    (300000, 64, "bf16", 16, 64, "cosine"),     # batch over a large store: sampled threshold
    (200003, 32, "f16", 5, 100, "ip"),
    (150001, 64, "bf16", 70, 16, "cosine"),     # two query groups
    (140000, 48, "bf16", 4, 1024, "cosine"),    # largest k
    (180001, 64, "f16", 8, 32, "ip"),           # filtered pass over 64-dim keys, inner product
    (262147, 64, "bf16", 40, 100, "cosine"),    # ... three query tiles, a ragged last wave
]


@pytest.mark.parametrize("case", SMALL_SCAN, ids=[str(i) for i in range(len(SMALL_SCAN))])
def test_short_key_scan_matches_oracle(case):
    n, d, kdt, nq, k, metric = case
    print(f"[short-scan] case={case}", flush=True)
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=n, d=d, key_dtype=kdt,
                     n_clusters=max(64, 2 * nq), n_outliers=2, metric=metric)
    ds = synth.make_datastore(w, 13, DEV)
    q, src = synth.make_queries(w, ds, 13, n_queries=nq)
    index = sense.sense_build_index(ds.keys, ds.spans, metric=metric)
    ids, sc, dr, _ = sense.sense_retrieve(index, q, k)
    torch.cuda.synchronize()
    o_s = oracle.scores(host_bits(ds.keys), kdt, q.cpu().numpy(), "f32", metric)
    for qq in range(nq):
        check_topk(ids[qq].cpu().numpy(), sc[qq].cpu().numpy(), o_s[qq], k)
    index.close()


def test_batched_short_keys_strided_store_equals_dense_copy():
    """64-dim keys at a row stride of 72 elements (144-byte rows, still
    16-byte aligned) take the same LDS-staged filtered pass as a dense
    store: the same ids and the same score bits as a dense copy of the
    keys, and the oracle's top k."""
    n, d, nq, k = 150_001, 64, 16, 64
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=n, d=d, key_dtype="bf16",
                     n_clusters=64, n_outliers=2, metric="cosine")
    ds = synth.make_datastore(w, 17, DEV, key_stride=72)
    assert ds.keys.stride(0) == 72
    q, _ = synth.make_queries(w, ds, 17, n_queries=nq)
    dense = ds.keys.contiguous()
    a = sense.sense_build_index(ds.keys, ds.spans, metric="cosine")
    b = sense.sense_build_index(dense, ds.spans, metric="cosine")
    ids_a, sc_a, _, _ = sense.sense_retrieve(a, q, k)
    ids_b, sc_b, _, _ = sense.sense_retrieve(b, q, k)
    torch.cuda.synchronize()
    assert torch.equal(ids_a, ids_b)
    assert torch.equal(sc_a.view(torch.int32), sc_b.view(torch.int32))
    o_s = oracle.scores(host_bits(dense), "bf16", q.cpu().numpy(), "f32", "cosine")
    for qq in range(nq):
        check_topk(ids_a[qq].cpu().numpy(), sc_a[qq].cpu().numpy(), o_s[qq], k)
    a.close()
    b.close()


def test_pca_retrieval_chain():
    """Project a 4096-dim store to 64 dims (bf16, normalised) and the query
    (fp32), search the projected store: against the oracle's own projection
    (rounded to bf16 by the host) and exact scan."""
    w = synth.scaled(synth.WORKLOADS["store-1m-d4096"], n=30000, n_clusters=120)
    ds = synth.make_datastore(w, 21, DEV)
    q, src = synth.make_queries(w, ds, 21)
    mean, basis = synth.make_pca_basis(ds, 21, 64)
    keys64 = sense.sense_project(ds.keys, basis, mean, True, out_dtype=torch.bfloat16)
    q64 = sense.sense_project(q, basis, mean, True, out_dtype=torch.float32)
    index = sense.sense_build_index(keys64, ds.spans)
    ids, sc, _, _ = sense.sense_retrieve(index, q64, 32)
    torch.cuda.synchronize()
    b = basis.cpu().numpy().astype(np.float64)
    mu = mean.cpu().numpy().astype(np.float64)
    ok = oracle.project(host_bits(ds.keys), "bf16", b, mu, True)
    ok_bits = torch.from_numpy(ok).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    oq = oracle.project(q.cpu().numpy(), "f32", b, mu, True).astype(np.float32)
    o_s = oracle.scores(ok_bits, "bf16", oq, "f32")
    check_topk(ids[0].cpu().numpy(), sc[0].cpu().numpy(), o_s[0], 32)
    assert int(ids[0, 0]) == int(src[0])
    index.close()


def test_batched_short_scan_when_every_row_passes_the_threshold():
    """Rows at the sample positions (multiples of n // 32768) point away from
    the queries and every other row points at them, so the sampled
    threshold is the lowest score and every row passes the filter: the
    result must still be the exact top-k (ties to the lower row)."""
    n, d = 200000, 64
    step = n // 32768
    g = torch.Generator(device=DEV).manual_seed(5)
    x = torch.randn(d, generator=g, device=DEV)
    keys = x.repeat(n, 1)
    keys[::step] = -x
    keys = keys.to(torch.bfloat16).contiguous()
    spans = torch.arange(n, dtype=torch.int32, device=DEV).unsqueeze(1).repeat(1, 4).contiguous()
    q = torch.stack([x * s for s in (1.0, 2.0, 0.5, 3.0)]).contiguous()
    index = sense.sense_build_index(keys, spans)
    ids, sc, dr, _ = sense.sense_retrieve(index, q, 64)
    torch.cuda.synchronize()
    want = [i for i in range(n) if i % step != 0][:64]
    for r in range(4):
        assert ids[r].cpu().tolist() == want
        assert dr[r, :, 0].cpu().tolist() == want
    o_s = oracle.scores(host_bits(keys[:200]), "bf16", q.cpu().numpy(), "f32", "cosine")
    np.testing.assert_allclose(sc[:, 0].cpu().numpy(), o_s[:, 1], rtol=1e-3)
    index.close()


def test_full_size_store_projection():
    """The store projection at the bench's shape: 1M x 4096 bf16 hidden
    states -> 64 bf16, normalised (matrix-core route), 512 seeded sample rows
    against the oracle; the 64 fp32 queries of the batched shape (direct
    route) in full."""
    w = synth.WORKLOADS["store-1m-pca64-q64"]
    seed = 1000 + list(synth.WORKLOADS).index(w.name)
    print(f"[project] full size n={w.n} d={w.d} -> {w.proj}", flush=True)
    ds = synth.make_datastore(w, seed, DEV)
    q, _ = synth.make_queries(w, ds, seed)
    mean, basis = synth.make_pca_basis(ds, seed, w.proj)
    keys64 = sense.sense_project(ds.keys, basis, mean, True, out_dtype=torch.bfloat16)
    q64 = sense.sense_project(q, basis, mean, True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(seed).choice(w.n, 512, replace=False))
    rows_t = torch.from_numpy(rows).to(DEV)
    check_projection(keys64[rows_t], host_bits(ds.keys[rows_t]), "bf16", basis, mean, True,
                     "bf16")
    check_projection(q64, q.cpu().numpy(), "f32", basis, mean, True, "f32")
    print("[project] sampled store rows and all queries ok", flush=True)
    del ds, keys64
    torch.cuda.empty_cache()


@pytest.mark.parametrize("nq", [1, 64])
def test_full_size_short_key_retrieval(nq):
    """Retrieval over a projected-shape store at the bench's size: 1M x 64
    bf16 keys, k = 64; one query takes the short-key scan, 64 the batched
    path with the sampled threshold.  Every query against the oracle's
    scores of all rows."""
    n, d, k = 1 << 20, 64, 64
    print(f"[short-scan] full size n={n} d={d} Q={nq} k={k}", flush=True)
    w = synth.scaled(synth.WORKLOADS["tiny-16k-d4096"], n=n, d=d, key_dtype="bf16", k=k,
                     n_clusters=4096, n_outliers=2)
    ds = synth.make_datastore(w, 53, DEV)
    q, src = synth.make_queries(w, ds, 53, n_queries=nq)
    index = sense.sense_build_index(ds.keys, ds.spans)
    ids, sc, dr, _ = sense.sense_retrieve(index, q, k)
    torch.cuda.synchronize()
    o_s = oracle.scores(host_bits(ds.keys), "bf16", q.cpu().numpy(), "f32")
    spans = ds.spans.cpu().numpy()
    for qq in range(nq):
        g_ids = ids[qq].cpu().numpy()
        check_topk(g_ids, sc[qq].cpu().numpy(), o_s[qq], k)
        assert np.array_equal(dr[qq].cpu().numpy(), oracle.gather(spans, None, g_ids)[0])
    print(f"[short-scan] {nq} queries ok", flush=True)
    index.close()
