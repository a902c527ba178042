"""Pins for the retrieval half of the oracle (exact scan, full-sort top-k, gather).

Each test checks the oracle against something other than itself: hand-worked
values (golden fixture), numpy's own float16 decoding and BLAS products with
lexsort, closed forms (a planted copy has cosine 1), and invariances of the
definition (cosine under positive power-of-two scaling, IP = cosine for unit
keys).  Sec. 3.1 Eq. 3, Sec. 3.2 Eqs. 7-8 and Alg. 2 define the computation.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def bf16_bits(x):
    """Round-to-nearest-even float32 -> bfloat16 bit patterns (test helper)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_to_f64(bits):
    with np.errstate(invalid="ignore"):
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f16_bits(x):
    return np.asarray(x, dtype=np.float16).view(np.uint16)


def test_tiny_datastore_golden_ip_and_cosine():
    g = json.load(open(os.path.join(GOLDEN, "tiny_datastore.json")))
    keys = f16_bits(np.array(g["keys"], dtype=np.float32))
    q = np.array(g["query"], dtype=np.float32)
    s_ip = oracle.scores(keys, "f16", q, "f32", metric="ip")[0]
    assert s_ip.tolist() == [float(v) for v in g["ip_scores"]]
    ids, _ = oracle.topk(s_ip, 7)
    assert ids.tolist() == g["ip_order"]
    s_cos = oracle.scores(keys, "f16", q, "f32", metric="cosine")[0]
    np.testing.assert_allclose(s_cos, g["cosine_scores"], rtol=1e-15, atol=1e-15)
    ids, sc = oracle.topk(s_cos, 4)
    assert ids.tolist() == g["cosine_order"][:4]
    spans = np.array(g["spans"], dtype=np.int32)
    dr, dl = oracle.gather(spans, np.array(g["span_len"], dtype=np.int32), ids)
    assert dr.tolist() == g["cosine_top4_drafts"]
    assert dl.tolist() == g["cosine_top4_draft_len"]


def test_same_keys_bf16_give_same_result():
    g = json.load(open(os.path.join(GOLDEN, "tiny_datastore.json")))
    keys = bf16_bits(np.array(g["keys"], dtype=np.float32))
    q = bf16_bits(np.array(g["query"], dtype=np.float32))
    s_ip = oracle.scores(keys, "bf16", q, "bf16", metric="ip")[0]
    assert s_ip.tolist() == [float(v) for v in g["ip_scores"]]


def test_f16_decoding_matches_numpy_on_every_pattern():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = oracle.decode(bits, "f16")
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zero is preserved
    assert np.signbit(got[0x8000]) and not np.signbit(got[0])


def test_bf16_decoding_matches_bit_shift_on_every_pattern():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bf16_to_f64(bits)
    got = oracle.decode(bits, "bf16")
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


@pytest.mark.parametrize("key_dtype", ["f16", "bf16"])
@pytest.mark.parametrize("metric", ["ip", "cosine"])
def test_against_numpy_matmul_and_lexsort(key_dtype, metric):
    rng = np.random.default_rng(7)
    n, d, stride = 3001, 40, 48
    kf = rng.normal(size=(n, stride)).astype(np.float32)
    kf[:, :3] *= 20.0                                    # outlier dims
    keys = f16_bits(kf) if key_dtype == "f16" else bf16_bits(kf)
    q = rng.normal(size=(2, d)).astype(np.float32)
    got = oracle.scores(keys, key_dtype, q, "f32", metric=metric, key_stride=stride, d=d)
    kd = (keys.view(np.float16).astype(np.float64) if key_dtype == "f16"
          else bf16_to_f64(keys))[:, :d]
    ref = q.astype(np.float64) @ kd.T
    if metric == "cosine":
        ref = ref / np.linalg.norm(q.astype(np.float64), axis=1)[:, None]
        ref = ref / np.linalg.norm(kd, axis=1)[None, :]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    for qi in range(2):
        order = np.lexsort((np.arange(n), -ref[qi]))
        ids, sc = oracle.topk(got[qi], 50)
        srt = np.sort(ref[qi])[::-1]
        assert np.min(np.abs(np.diff(srt[:51]))) > 1e-9    # no near-ties at this seed
        assert ids.tolist() == order[:50].tolist()


def test_planted_copy_ranks_first_with_cosine_one():
    rng = np.random.default_rng(3)
    n, d = 2000, 64
    kf = rng.normal(size=(n, d)).astype(np.float32) * rng.uniform(0.1, 10, size=(n, 1)).astype(np.float32)
    keys = bf16_bits(kf)
    for r in (0, 777, n - 1):
        q = bf16_to_f64(keys[r]).astype(np.float32)       # exact copy of stored row
        s = oracle.scores(keys, "bf16", q, "f32", metric="cosine")[0]
        ids, sc = oracle.topk(s, 3)
        assert ids[0] == r
        assert abs(sc[0] - 1.0) < 1e-15


def test_duplicates_tie_by_lower_index_and_zero_rows_score_zero():
    base = np.array([[1.0, 2.0, 3.0, 4.0]], dtype=np.float32)
    kf = np.repeat(base, 5, axis=0)
    kf[2] = 0.0
    keys = f16_bits(kf)
    q = np.array([1.0, 1.0, 1.0, 1.0], dtype=np.float32)
    for metric in ("ip", "cosine"):
        s = oracle.scores(keys, "f16", q, "f32", metric=metric)[0]
        assert s[2] == 0.0
        ids, _ = oracle.topk(s, 5)
        assert ids.tolist() == [0, 1, 3, 4, 2]


def test_cosine_invariant_under_power_of_two_scaling():
    rng = np.random.default_rng(11)
    n, d = 500, 32
    kf = rng.normal(size=(n, d)).astype(np.float32)
    q = rng.normal(size=(1, d)).astype(np.float32)
    keys = f16_bits(kf)
    scaled = f16_bits(kf.astype(np.float16).astype(np.float32) * np.where(np.arange(n) % 2, 4.0, 2.0)[:, None])
    a = oracle.scores(keys, "f16", q, "f32", metric="cosine")[0]
    b = oracle.scores(scaled, "f16", q, "f32", metric="cosine")[0]
    np.testing.assert_allclose(a, b, rtol=1e-14, atol=1e-15)


def test_ip_equals_cosine_for_unit_rows_and_unit_query():
    # rows with exactly one +-1 entry have norm 1 exactly
    rng = np.random.default_rng(5)
    n, d = 300, 16
    kf = np.zeros((n, d), dtype=np.float32)
    kf[np.arange(n), rng.integers(0, d, n)] = rng.choice([-1.0, 1.0], n)
    q = np.zeros((1, d), dtype=np.float32)
    q[0, 3] = 1.0
    keys = f16_bits(kf)
    a = oracle.scores(keys, "f16", q, "f32", metric="ip")
    b = oracle.scores(keys, "f16", q, "f32", metric="cosine")
    assert np.array_equal(a, b)


def test_nan_scores_sort_last_and_k_beyond_n():
    s = np.array([0.5, np.nan, 2.0, -1.0, np.nan, 2.0])
    ids, sc = oracle.topk(s, 8)
    assert ids.tolist()[:4] == [2, 5, 0, 3]
    assert ids.tolist()[4:6] == [1, 4]          # NaN rows last, among themselves by row
    assert ids.tolist()[6:] == [-1, -1]


def test_gather_is_indexing():
    rng = np.random.default_rng(2)
    spans = rng.integers(0, 32000, size=(100, 9)).astype(np.int32)
    lens = rng.integers(0, 10, size=100).astype(np.int32)
    ids = rng.permutation(100)[:17].astype(np.int64)
    dr, dl = oracle.gather(spans, lens, ids)
    for r, i in enumerate(ids):
        assert dl[r] == lens[i]
        assert dr[r, :lens[i]].tolist() == spans[i, :lens[i]].tolist()
        assert (dr[r, lens[i]:] == -1).all()
    dr2, dl2 = oracle.gather(spans, None, ids)
    assert np.array_equal(dr2, spans[ids]) and (dl2 == 9).all()
