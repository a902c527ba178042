"""Pins for the inverted-file oracle (the ANN retriever of Sec. 3.2 Eq. 7 as
the implementation details configure it: a coarse quantizer with nprobe
lists searched, product-quantized residuals): probing every list reduces
IVF-Flat to the exact search; a numpy re-implementation of probe-then-rank
agrees; data built from codebook entries is encoded exactly and scored
exactly by the asymmetric distance; planted rows join their own list; ties
go to the lower id; the k-th best score never falls as nprobe grows."""
import numpy as np
import pytest
import torch

import oracle


def bits(x, dt):
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    t = t.to(torch.bfloat16 if dt == "bf16" else torch.float16)
    return t.view(torch.int16).numpy().view(np.uint16), t.float().numpy().astype(np.float64)


def clustered(rng, n, d, nlist, dt="bf16"):
    cen = rng.normal(0, 1, (nlist, d))
    lab = rng.integers(0, nlist, n)
    x = cen[lab] + rng.normal(0, 0.4, (n, d))
    b, dec = bits(x, dt)
    return b, dec, cen


@pytest.mark.parametrize("metric", ["ip", "cosine"])
def test_probing_every_list_is_the_exact_search(metric):
    rng = np.random.default_rng(0)
    kb, _, cen = clustered(rng, 3000, 32, 20)
    lists, _ = oracle.ivf_assign(kb, "bf16", cen, metric)
    q = rng.normal(0, 1, 32).astype(np.float32)
    probe, _, ids, sc = oracle.ivf_search(q, cen, lists, 20, 25, metric, keys=kb)
    exact = oracle.scores(kb, "bf16", q[None], "f32", metric)[0]
    e_ids, e_sc = oracle.topk(exact, 25)
    assert np.array_equal(ids, e_ids)
    assert np.array_equal(sc, e_sc)
    assert sorted(probe.tolist()) == list(range(20))


@pytest.mark.parametrize("metric", ["ip", "cosine"])
def test_probe_then_rank_matches_numpy(metric):
    rng = np.random.default_rng(1)
    kb, dec, cen = clustered(rng, 4000, 24, 50)
    lists, _ = oracle.ivf_assign(kb, "bf16", cen, metric)
    for s in range(5):
        q = rng.normal(0, 1, 24)
        probe, coarse, ids, sc = oracle.ivf_search(q, cen, lists, 7, 30, metric, keys=kb)
        cs = cen @ q
        ks = dec @ q
        if metric == "cosine":
            cs = cs / (np.linalg.norm(cen, axis=1) * np.linalg.norm(q))
            ks = ks / (np.linalg.norm(dec, axis=1) * np.linalg.norm(q))
        np.testing.assert_allclose(coarse, cs, rtol=1e-12)
        want_probe = np.lexsort((np.arange(50), -cs))[:7]
        assert probe.tolist() == want_probe.tolist()
        rows = np.flatnonzero(np.isin(lists, want_probe))
        order = rows[np.lexsort((rows, -ks[rows]))][:30]
        assert ids.tolist() == order.tolist()
        np.testing.assert_allclose(sc, ks[order], rtol=1e-12)


def pq_planted(rng, n, d, nlist, m, ksub):
    """Keys = centroid + concatenated codebook entries, all multiples of 1/8
    in a small range, so every key is exact in bf16 and every residual slice
    is exactly one codebook entry."""
    dsub = d // m
    cen = rng.integers(-8, 9, (nlist, d)) / 8.0
    cb = rng.integers(-4, 5, (m, ksub, dsub)) / 8.0
    # distinct codebook entries so the nearest entry is unique
    for j in range(m):
        _, first = np.unique(cb[j], axis=0, return_index=True)
        keep = np.zeros(ksub, bool)
        keep[first] = True
        cb[j][~keep] = 5.0 + np.arange((~keep).sum())[:, None] / 8.0
    lab = rng.integers(0, nlist, n)
    codes = rng.integers(0, ksub, (n, m)).astype(np.uint8)
    x = cen[lab] + np.concatenate([cb[j][codes[:, j]] for j in range(m)], axis=1)
    kb, dec = bits(x, "bf16")
    assert np.array_equal(dec, x)
    return kb, cen, cb, lab.astype(np.int32), codes


def test_pq_of_planted_data_is_exact():
    rng = np.random.default_rng(2)
    kb, cen, cb, lab, codes = pq_planted(rng, 1500, 16, 12, 4, 32)
    got = oracle.pq_encode(kb, "bf16", cen, lab, cb)
    assert np.array_equal(got, codes)
    q = rng.normal(0, 1, 16)
    for nprobe in (3, 12):
        _, _, ids_pq, sc_pq = oracle.ivf_search(q, cen, lab, nprobe, 40, "ip", codes=codes,
                                                codebooks=cb)
        _, _, ids_f, sc_f = oracle.ivf_search(q, cen, lab, nprobe, 40, "ip", keys=kb)
        np.testing.assert_allclose(sc_pq, sc_f, rtol=1e-12, atol=1e-12)
        assert np.array_equal(ids_pq, ids_f)


def test_pq_score_is_normalised_query_dot_reconstruction():
    rng = np.random.default_rng(3)
    kb, cen, cb, lab, codes = pq_planted(rng, 500, 16, 6, 4, 16)
    q = rng.normal(0, 1, 16) * 3.0
    _, _, ids, sc = oracle.ivf_search(q, cen, lab, 6, 10, "cosine", codes=codes, codebooks=cb)
    rec = cen[lab] + np.concatenate([cb[j][codes[:, j]] for j in range(4)], axis=1)
    want = rec @ (q / np.linalg.norm(q))
    order = np.lexsort((np.arange(500), -want))[:10]
    assert ids.tolist() == order.tolist()
    np.testing.assert_allclose(sc, want[order], rtol=1e-12)


def test_assign_planted_rows_and_ties():
    rng = np.random.default_rng(4)
    cen = rng.normal(0, 1, (30, 16))
    cen[7] = cen[3]                                  # duplicate centroid: lower id wins
    lab = rng.integers(0, 30, 400)
    x = cen[lab] + rng.normal(0, 1e-3, (400, 16))
    kb, _ = bits(x, "f16")
    lists, _ = oracle.ivf_assign(kb, "f16", cen, "cosine")
    want = np.where(lab == 7, 3, lab)
    assert np.array_equal(lists, want)


def test_encode_ties_go_to_the_lower_entry():
    cen = np.zeros((1, 4))
    cb = np.zeros((2, 3, 2))
    cb[0] = [[1, 0], [0.5, 0.5], [1, 0]]             # entries 0 and 2 equal
    cb[1] = [[0, 0], [0, 0], [2, 2]]
    kb, _ = bits(np.array([[1, 0, 0, 0], [0.5, 0.5, 2, 2]]), "bf16")
    codes = oracle.pq_encode(kb, "bf16", cen, np.zeros(2, np.int32), cb)
    assert codes.tolist() == [[0, 0], [1, 2]]


def test_kth_score_never_falls_as_nprobe_grows():
    rng = np.random.default_rng(5)
    kb, _, cen = clustered(rng, 2000, 16, 40)
    lists, _ = oracle.ivf_assign(kb, "bf16", cen, "cosine")
    q = rng.normal(0, 1, 16)
    prev = None
    for nprobe in (1, 2, 4, 8, 16, 40):
        _, _, ids, sc = oracle.ivf_search(q, cen, lists, nprobe, 20, "cosine", keys=kb)
        sc = np.where(np.isnan(sc), -np.inf, sc)
        if prev is not None:
            assert np.all(sc >= prev)
        prev = sc
