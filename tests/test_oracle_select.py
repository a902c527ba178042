"""Pins for the candidate-selection oracle (Sec. 3.2 Eq. 8; Alg. 2 composite
score, Top-N, dynamic boost delta and anchor override): a hand-worked golden
example, the lexicographic order that alpha >> beta imposes, the pure
similarity order at alpha = 0 (numpy lexsort), the delta boost, position
tie-breaks and the override's guarantee."""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_example():
    g = json.load(open(os.path.join(GOLDEN, "candidate_selection_example.json")))
    dr, ln, src, sc = oracle.select_candidates(
        np.array(g["static_scores"]), np.array(g["static_drafts"]), np.array(g["static_len"]),
        g["anchor"], g["top_n"], g["alpha"], g["beta"], g["delta"],
        scores_d=np.array(g["dynamic_scores"]), drafts_d=np.array(g["dynamic_drafts"]),
        len_d=np.array(g["dynamic_len"]))
    assert src.tolist() == g["expected_source"]
    np.testing.assert_allclose(sc, g["expected_scores"], rtol=0, atol=1e-12)
    assert dr.tolist() == g["expected_drafts"]
    assert ln.tolist() == g["expected_len"]
    _, _, src_all, sc_all = oracle.select_candidates(
        np.array(g["static_scores"]), np.array(g["static_drafts"]), np.array(g["static_len"]),
        g["anchor"], 7, g["alpha"], g["beta"], g["delta"], anchor_override=False,
        scores_d=np.array(g["dynamic_scores"]), drafts_d=np.array(g["dynamic_drafts"]),
        len_d=np.array(g["dynamic_len"]))
    assert src_all.tolist() == g["order"]
    np.testing.assert_allclose(sc_all, np.array(g["composite_all"])[g["order"]], atol=1e-12)


def _random(rng, n, m=6, vocab=20):
    s = rng.uniform(-1, 1, n)
    d = rng.integers(0, vocab, (n, m)).astype(np.int32)
    ln = rng.integers(0, m + 1, n).astype(np.int32)
    for i in range(n):
        d[i, ln[i]:] = -1
    return s, d, ln


def test_alpha_much_larger_than_beta_is_lexicographic():
    rng = np.random.default_rng(3)
    s, d, ln = _random(rng, 200)
    anchor = 4
    dr, _, src, _ = oracle.select_candidates(s, d, ln, anchor, 50, 1e6, 1.0, anchor_override=False)
    match = (ln > 0) & (d[:, 0] == anchor)
    ref = sorted(range(200), key=lambda i: (not match[i], -s[i], i))[:50]
    assert src.tolist() == ref


def test_alpha_zero_is_similarity_order_over_both_sources():
    rng = np.random.default_rng(5)
    s, d, ln = _random(rng, 120)
    sd_, dd, ld = _random(rng, 40)
    delta = 0.25
    _, _, src, _ = oracle.select_candidates(s, d, ln, 1, 60, 0.0, 1.0, delta,
                                            anchor_override=False, scores_d=sd_, drafts_d=dd,
                                            len_d=ld)
    allsc = np.concatenate([s, sd_ + delta])
    ref = np.lexsort((np.arange(160), -allsc))[:60]
    assert src.tolist() == ref.tolist()


def test_large_delta_puts_dynamic_hits_first():
    rng = np.random.default_rng(8)
    s, d, ln = _random(rng, 30)
    sd_, dd, ld = _random(rng, 10)
    _, _, src, _ = oracle.select_candidates(s, d, ln, 1, 12, 0.0, 1.0, 100.0,
                                            anchor_override=False, scores_d=sd_, drafts_d=dd,
                                            len_d=ld)
    assert sorted(src.tolist()[:10]) == list(range(30, 40))


def test_equal_scores_keep_position_order():
    s = np.full(6, 0.5)
    d = np.tile(np.arange(4, dtype=np.int32), (6, 1))
    _, _, src, _ = oracle.select_candidates(s, d, None, 99, 6, 1.0, 1.0, anchor_override=False,
                                            scores_d=np.full(3, 0.5), drafts_d=d[:3])
    assert src.tolist() == [0, 1, 2, 3, 4, 5]


@pytest.mark.parametrize("top_n", [1, 2, 7])
def test_override_puts_the_anchor_first_in_first_and_last_row(top_n):
    rng = np.random.default_rng(top_n)
    s, d, ln = _random(rng, 20)
    anchor = 17
    dr0, ln0, src0, _ = oracle.select_candidates(s, d, ln, anchor, top_n, 0.0, 1.0,
                                                 anchor_override=False)
    dr, lns, src, _ = oracle.select_candidates(s, d, ln, anchor, top_n, 0.0, 1.0)
    assert np.array_equal(src, src0)
    assert dr[0, 0] == anchor and dr[-1, 0] == anchor
    assert lns[0] >= 1 and lns[-1] >= 1
    assert np.array_equal(dr[1:-1], dr0[1:-1])
    assert np.array_equal(dr[:, 1:], dr0[:, 1:])


def test_binary32_mode_orders_like_the_f64_mode_when_scores_are_apart():
    g = json.load(open(os.path.join(GOLDEN, "candidate_selection_example.json")))
    args = (np.array(g["static_scores"]), np.array(g["static_drafts"]), np.array(g["static_len"]),
            g["anchor"], g["top_n"], g["alpha"], g["beta"], g["delta"])
    kw = dict(scores_d=np.array(g["dynamic_scores"]), drafts_d=np.array(g["dynamic_drafts"]),
              len_d=np.array(g["dynamic_len"]))
    dr, ln, src, sc = oracle.select_candidates(*args, precision="f32", **kw)
    assert src.tolist() == g["expected_source"]
    assert dr.tolist() == g["expected_drafts"]
    np.testing.assert_allclose(sc, g["expected_scores"], rtol=1e-6)
    assert np.array_equal(sc.astype(np.float32).astype(np.float64), sc)


def test_binary32_mode_ties_scores_that_round_together():
    s = np.array([0.5, 0.5 + 1e-12])
    d = np.array([[1, 2], [3, 4]], dtype=np.int32)
    _, _, src64, _ = oracle.select_candidates(s, d, None, 9, 2, 0.0, 1.0, anchor_override=False)
    _, _, src32, _ = oracle.select_candidates(s, d, None, 9, 2, 0.0, 1.0, anchor_override=False,
                                              precision="f32")
    assert src64.tolist() == [1, 0]
    assert src32.tolist() == [0, 1]


def test_dynamic_spans_are_the_following_tokens():
    spans, lens = oracle.dynamic_spans([5, 6, 7, 8], 3)
    assert spans.tolist() == [[5, 6, 7], [6, 7, 8], [7, 8, -1], [8, -1, -1]]
    assert lens.tolist() == [3, 3, 2, 1]


def test_override_gives_the_first_and_last_draft_an_accepted_token():
    """Alg. 2's override forces both ends of the pool to start with the greedy
    anchor, and row 0 of every draft is judged by the shared distribution
    whose argmax is that anchor, so the exact-match gate accepts it."""
    rng = np.random.default_rng(11)
    vocab, m, n = 50, 5, 12
    s, d, ln = _random(rng, n, m=m, vocab=vocab)
    shared = rng.normal(0, 2, vocab).astype(np.float32)
    anchor = int(np.argmax(shared))
    top_n = 6
    dr, lns, _, _ = oracle.select_candidates(s, d, ln, anchor, top_n, 0.0, 1.0)
    logits = rng.normal(0, 2, (top_n, m, vocab)).astype(np.float32)
    logits[:, 0, :] = shared
    out = oracle.soft_gate_verify(logits, "f32", dr, lns, gamma=10.0)
    assert out["accept_len"][0] >= 1 and out["accept_len"][-1] >= 1


def test_empty_draft_gets_no_anchor_bonus():
    """I(s[0] = anchor) needs a first token: a continuation of length 0 has
    none, so its composite score is beta * s even when its stored row starts
    with the anchor."""
    s = np.array([0.5, 0.25])
    d = np.array([[9, 1, 2], [9, 3, 4]], dtype=np.int32)
    ln = np.array([0, 2], dtype=np.int32)
    _, _, src, sc = oracle.select_candidates(s, d, ln, 9, 2, 10.0, 1.0, anchor_override=False)
    assert src.tolist() == [1, 0]
    assert sc.tolist() == [10.25, 0.5]
